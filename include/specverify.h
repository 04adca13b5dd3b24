/*
 * specverify.h — C ABI of the MI355X (gfx950) speculative-verification and
 * TV-loss library (libspecverify.so).
 *
 * Method: "Breaking Entropy Bounds: Accelerating RL Training via MTP with
 * Rejection Sampling".  Sec. 2.2 (Eq. reject_sample) and App. G.1 (Alg.
 * rs_multinomial) define chain rejection-sampling verification of K draft
 * tokens; Sec. 4.1 (Eqs. tv_loss, tv_grad), App. A and Sec. 4.2 (Eq. e2e_tv)
 * define the TV loss, its gradient and the end-to-end multi-step TV loss.
 * Sec. 2.2 (Eq. target_only) defines target-only verification, App. G.1 the
 * draft-stage sampler, Sec. 3 and App. E the acceptance diagnostics, App. G.2
 * (Alg. rs_gumbel) Gumbel-max verification and the Gumbel-max draft sampler;
 * Sec. 4.1 (footnote), Table grad_comparison, App. B and App. C the CE and KL
 * objectives the TV loss is compared against.
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The
 *    library allocates no device or host memory and keeps no mutable state
 *    between calls other than what lives in the caller's workspace.
 *  - The last dimension (vocabulary, length V) must be contiguous.  Other
 *    dimensions take element strides (>= 0), so shifted views of larger
 *    tensors can be passed without copies.  A tensor whose last element,
 *    reached through the strides, lies beyond the 64-bit address space is
 *    SPEC_EINVAL.
 *  - Work is only enqueued on `stream` (a hipStream_t passed as void*, NULL =
 *    the null stream); no call synchronises with the host.
 *  - Host-checkable argument errors are returned synchronously before any
 *    work is enqueued.  Misaligned pointers or strides are not an error:
 *    they select element-wise loads instead of 16-byte vector loads.
 *  - The workspace is scratch memory: it needs no initialisation, each call
 *    overwrites what it reads, and no state is carried from one call to the
 *    next.  Calls that share a workspace must not run concurrently (enqueue
 *    them on one stream).
 *  - Each call is a short fixed sequence of kernel launches on `stream`
 *    (spec_verify: 4, or 3 on its single-read path; spec_tv_loss_fwd_bwd:
 *    5, or 6 with a gradient; spec_verify_target_only: 2, spec_sample: 2,
 *    spec_diagnostics: 4, spec_verify_gumbel: 5, or 4 without overlaps,
 *    spec_sample_gumbel: 2, spec_kl_loss_fwd_bwd: 5, or 6 with a gradient,
 *    one more for reverse KL).
 *    Only the single-read path of spec_verify has
 *    workgroups that wait for other workgroups of the same launch; it is a
 *    cooperative launch (all its workgroups resident at once) and every wait
 *    is bounded.  No other launch waits on another workgroup.
 *  - Entry points are thread-safe; each call is independent.
 *  - Logits are bfloat16 (raw 16-bit patterns) or float32.  Arithmetic is
 *    float32 per element with float64 accumulation across vectors, threads
 *    and workgroups.
 */
#ifndef SPECVERIFY_H
#define SPECVERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEC_VERSION 2

/* The enumerations below are int-sized.  C++ gives them int as their fixed
 * underlying type, so that any int a caller passes (a C program, a foreign
 * function interface) is a value of the type and the library's range checks
 * see it; C declares them without one. */
#ifdef __cplusplus
#define SPEC_ENUM_INT : int
#else
#define SPEC_ENUM_INT
#endif
#define SPEC_MAX_K 8 /* largest number of draft steps K */
/* largest vocabulary V (2^31 - 2^16): element indices are 32-bit and run one
 * 16384-element chunk past V where a row's last chunk is rounded up */
#define SPEC_MAX_V 2147418112

typedef enum SPEC_ENUM_INT { SPEC_F32 = 0, SPEC_BF16 = 1 } spec_dtype;

typedef enum SPEC_ENUM_INT {
  SPEC_OK = 0,
  SPEC_EINVAL = 1,       /* bad pointer, size, stride, temperature, mode */
  SPEC_EUNSUPPORTED = 2, /* dtype or K outside what the library handles */
  SPEC_EWORKSPACE = 4,   /* workspace NULL or smaller than *_workspace_size */
  SPEC_EHIP = 5          /* the HIP runtime reported an error (launch, device query) */
} spec_status;

typedef enum SPEC_ENUM_INT {
  SPEC_TV_E2E = 0,     /* Sec. 4.2 Eq. e2e_tv: L = 1 - (1/K) sum_j prod_{i<=j} alpha_i        */
  SPEC_TV_PROD = 1,    /* L = -prod_k alpha_k (negated probability that all K drafts pass)  */
  SPEC_TV_PER_STEP = 2 /* Sec. 4.1 Eq. tv_loss averaged over steps: (1/K) sum_k (1 - alpha_k) */
} spec_tv_mode;

/* Bytes of workspace spec_verify needs for this shape (0 on invalid sizes). */
size_t spec_verify_workspace_size(int B, int K, int V, spec_dtype dtype);

/*
 * spec_verify — chain rejection-sampling verification of K draft tokens for B
 * independent batch rows (Sec. 2.2 Eq. reject_sample; App. G.1 Alg.
 * rs_multinomial).
 *
 * For row b, with T = temperature[b] (or temperature_scalar):
 *   p_i = softmax(target[b, i, :] / T), i = 0..K (row K: bonus position after the last draft)
 *   q_i = softmax(draft[b, i, :] / T),  i = 0..K-1
 *   step i accepts x_i = draft_ids[b, i] iff u_i * q_i(x_i) < p_i(x_i)
 *   n = first rejected step (K if none); accept_len[b] = n
 *   emitted[b, 0..n-1] = x_0..x_{n-1}
 *   emitted[b, n] = smallest v with C(v) > u' * Z, C = cumulative sum (vocabulary
 *       order) of r = max(0, p_n - q_n) if n < K, else of r = p_K; Z = sum r
 *       (if Z is exactly 0 the sample is drawn from p_n)
 *   emitted[b, n+1..K] = -1
 *   overlap[b, i] = sum_v min(p_i(v), q_i(v)) = 1 - d_TV(p_i, q_i) for every i < K
 * Uniforms: block = Philox4x64-10(counter = (b, i, offset, 0), key = (seed, 0))
 *   (Salmon et al., SC'11); u_i = (word0 >> 40) * 2^-24, the resample uniform of
 *   the emitting step n is (word1 >> 40) * 2^-24 of the block at (b, n).
 *
 * target_logits  [B, K+1, V] element strides (t_stride_b, t_stride_k), dtype
 * draft_logits   [B, K,   V] element strides (d_stride_b, d_stride_k), dtype
 * draft_ids      [B, K] int32, contiguous; ids sampled from q_i
 * temperature    [B] float32 device array, or NULL to use temperature_scalar
 *                (which must then be finite and > 0)
 * accept_len     [B] int32 out
 * emitted_ids    [B, K+1] int32 out, contiguous
 * overlap        [B, K] float32 out, or NULL (then the overlaps of the
 *                accepted steps are not formed)
 * p_at_draft, q_at_draft  [B, K] float32 out: p_i(x_i), q_i(x_i) (may be NULL)
 * logz_target    [B, K+1] float32 out: natural-log partition function of z/T (may be NULL)
 * logz_draft     [B, K]   float32 out (may be NULL)
 * workspace      device memory of at least spec_verify_workspace_size bytes
 *
 * Row data errors (NaN or +inf logits, a row that is all -inf, a draft id
 * outside [0, V), a per-row temperature that is not finite and > 0) do not
 * fail the call: that row gets accept_len = -1, emitted = -1 and NaN in every
 * float output.  -inf logits are legal (probability 0).
 * Limits: 1 <= K <= SPEC_MAX_K, 1 <= V <= SPEC_MAX_V, 1 <= B, B*(K+1) < 2^31.
 *
 * Two launch paths compute the same method (spec_verify takes the chain;
 * spec_verify_ex selects either):
 *  - single read (K <= 4, 16-byte aligned rows, V a multiple of 8 for bf16
 *    or of 4 for fp32, at most 64 slices of 4096 bf16 / 2048 fp32 elements
 *    per row): each batch row is spread over a
 *    group of workgroups, one per slice, which keep their slice of all 2K+1
 *    rows in registers and LDS, exchange the slice statistics through the
 *    workspace and take the overlaps and residual sums without reading the
 *    logits again; then one launch per batch row picks the resampled token
 *    (reading one slice of one row pair again);
 *  - chain (every shape): statistics, decision, a second read of the draft
 *    pairs (only each batch row's residual step without `overlap`), then the
 *    same per-row launch.
 * Either path forms each element's p - q for the residual from the exact
 * logit difference, with the two rows' normalisations reconciled, so that
 * the residual distribution matches exact arithmetic where p and q nearly
 * coincide.
 * Tokens are bit-exact functions of the inputs, seed and offset for either
 * path and any number of groups; the two paths' float32 normaliser sums differ
 * in summation order, which can move a decision only where its uniform lies
 * within float32 rounding of a decision boundary.
 */
spec_status spec_verify(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                        const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                        spec_dtype dtype, int B, int K, int V,
                        const int32_t* draft_ids,
                        const float* temperature, float temperature_scalar,
                        uint64_t seed, uint64_t offset,
                        int32_t* accept_len, int32_t* emitted_ids,
                        float* overlap, float* p_at_draft, float* q_at_draft,
                        float* logz_target, float* logz_draft,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Launch controls for spec_verify_ex (tests, benchmarks and tuning). */
typedef enum SPEC_ENUM_INT {
  SPEC_PATH_AUTO = 0,        /* the library's choice (the chain on MI355X)        */
  SPEC_PATH_CHAIN = 1,       /* always the four-launch chain                        */
  SPEC_PATH_SINGLE_READ = 2  /* single read; SPEC_EUNSUPPORTED where it does not qualify */
} spec_path;
typedef struct {
  int path;   /* spec_path */
  int groups; /* single read: number of workgroup groups (0 = chosen by the library;
                 more than the device holds at once selects the chain, or
                 SPEC_EUNSUPPORTED with SPEC_PATH_SINGLE_READ) */
  int residual_shape; /* chain: how the second pass reads each row's residual step
                         (0 = chosen by the library from B and V; 1 = one wave
                         per sub-chunk; 2 = one workgroup per sub-chunk, the
                         small-batch shape).  Every shape gives the same bits. */
} spec_launch;

/*
 * spec_verify_ex — spec_verify with explicit launch controls (NULL = the
 * defaults of spec_verify).  Same arguments, outputs and errors as
 * spec_verify; SPEC_EINVAL for an unknown path or residual shape, or a
 * negative group count.
 */
spec_status spec_verify_ex(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                           const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                           spec_dtype dtype, int B, int K, int V,
                           const int32_t* draft_ids,
                           const float* temperature, float temperature_scalar,
                           uint64_t seed, uint64_t offset,
                           int32_t* accept_len, int32_t* emitted_ids,
                           float* overlap, float* p_at_draft, float* q_at_draft,
                           float* logz_target, float* logz_draft,
                           void* workspace, size_t workspace_bytes, void* stream,
                           const spec_launch* launch);

/*
 * spec_verify_noalloc — spec_verify for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same arguments without the workspace, which is
 * instead a device array inside the library, one per GPU, held until the
 * process ends.  The call itself allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); the first call on a device looks up that
 * device's copy of the array.
 * Returns SPEC_EWORKSPACE when the shape needs more than
 * spec_verify_noalloc_max_workspace() bytes (32 MiB: every shape up to
 * B = 1024, K = 3, V = 262144 bf16 fits), and otherwise the statuses of
 * spec_verify.  Calls on one GPU share its array: calls that overlap in time
 * on one GPU (other streams, other host threads) race and must not be
 * issued; calls queued on one stream are safe.
 */
spec_status spec_verify_noalloc(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                                const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                                spec_dtype dtype, int B, int K, int V,
                                const int32_t* draft_ids,
                                const float* temperature, float temperature_scalar,
                                uint64_t seed, uint64_t offset,
                                int32_t* accept_len, int32_t* emitted_ids,
                                float* overlap, float* p_at_draft, float* q_at_draft,
                                float* logz_target, float* logz_draft, void* stream);

/* Largest workspace (bytes) spec_verify_noalloc can hold. */
size_t spec_verify_noalloc_max_workspace(void);

/* Bytes of workspace spec_tv_loss_fwd_bwd needs (0 on invalid sizes).  It
 * includes about one bit per logit (N*K*ceil(V/16384)*2048 bytes, about 1/32
 * of the gradient): the indicator 1[q <= p] of the forward pass, which the
 * gradient pass reads instead of the target logits. */
size_t spec_tv_workspace_size(int N, int K, int V, spec_dtype dtype);

/*
 * spec_tv_loss_fwd_bwd — fused TV-loss forward and gradient w.r.t. the draft
 * logits (Sec. 4.1 Eqs. tv_loss / tv_grad, App. A, App. F; Sec. 4.2 Eq. e2e_tv).
 *
 * For position n and draft step k:
 *   p = softmax(target[n, k, :] / T) (detached), q = softmax(draft[n, k, :] / T)
 *   alpha[n, k] = sum_v min(p_v, q_v),  S[n, k] = sum_v 1[q_v <= p_v] q_v
 *   L_n by `mode` (see spec_tv_mode); g[n, k] = d L_n / d alpha[n, k]
 *   loss = scale * sum_n L_n
 *   grad_draft[n, k, j] = scale * g[n, k] * (1/T) * q_j * (1[q_j <= p_j] - S[n, k])
 *
 * target_logits, draft_logits  [N, K, V], element strides (stride_n, stride_k)
 * temperature    finite and > 0 (one value for all positions)
 * loss           [1] float32 out (device)
 * overlap        [N, K] float32 out (may be NULL)
 * grad_draft     [N, K, V] float32 out, contiguous; NULL = forward only
 * NaN or infinite logits propagate as NaN into that position's loss and
 * gradient (no per-position status).
 * Limits: 1 <= K <= SPEC_MAX_K, 1 <= V <= SPEC_MAX_V, 1 <= N, N*K < 2^31.
 */
spec_status spec_tv_loss_fwd_bwd(const void* target_logits, int64_t t_stride_n, int64_t t_stride_k,
                                 const void* draft_logits, int64_t d_stride_n, int64_t d_stride_k,
                                 spec_dtype dtype, int N, int K, int V,
                                 float temperature, spec_tv_mode mode, float scale,
                                 float* loss, float* overlap, float* grad_draft,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spec_verify_gumbel needs (0 on invalid sizes). */
size_t spec_verify_gumbel_workspace_size(int B, int K, int V, spec_dtype dtype);

/*
 * spec_verify_gumbel — chain rejection-sampling verification with the
 * token at the emitting position drawn by the Gumbel-max trick (App. G.2,
 * Alg. rs_gumbel).  Arguments, outputs, accept tests, uniforms of the accept
 * tests and row-error handling are those of spec_verify; only emitted[b, n]
 * differs:
 *   emitted[b, n] = argmax_v [ log r(v) + G_v ],  r = max(0, p_n - q_n) if n < K,
 *                   and log r replaced by z_K / T for the bonus (n = K);
 *                   first index among ties; r = p_n if the residual has no mass
 *   G_v = -log(-log U_v), U_v = (bits + 1/2) * 2^-24, bits = the top 24 bits
 *         (v even) or bits 8..31 (v odd) of word (v >> 1) & 3 of
 *         Philox4x64-10(counter = (b, v >> 3, offset, 2), key = (seed, 0))
 * With overlap == NULL the pairs are not read a second time; the emitting
 * row (pair) is then the only one read again, in full.
 */
spec_status spec_verify_gumbel(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                               const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                               spec_dtype dtype, int B, int K, int V,
                               const int32_t* draft_ids,
                               const float* temperature, float temperature_scalar,
                               uint64_t seed, uint64_t offset,
                               int32_t* accept_len, int32_t* emitted_ids,
                               float* overlap, float* p_at_draft, float* q_at_draft,
                               float* logz_target, float* logz_draft,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spec_sample_gumbel needs (0 on invalid sizes). */
size_t spec_sample_gumbel_workspace_size(int R, int V, spec_dtype dtype);

/*
 * spec_sample_gumbel — the Gumbel-max draft stage (App. G.2): row r with
 * T = temperature[r] (or temperature_scalar) > 0 gets
 *   tokens[r] = argmax_v [ logits[r, v] / T + G_v ] (first index among ties),
 * G_v as in spec_verify_gumbel with counter (r, v >> 3, offset, 3); T == 0
 * takes the greedy token (first index of the largest logit).  One read of
 * the logits, no normaliser.
 * logits [R, V] with row stride stride_r; temperature [R] or NULL (scalar,
 * finite, >= 0); tokens [R] int32 out.  Row data errors (NaN or +inf
 * logits, all -inf, a negative or non-finite per-row temperature) give -1.
 * Limits: 1 <= R, 1 <= V <= SPEC_MAX_V.
 */
spec_status spec_sample_gumbel(const void* logits, int64_t stride_r, spec_dtype dtype, int R, int V,
                               const float* temperature, float temperature_scalar,
                               uint64_t seed, uint64_t offset, int32_t* tokens,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spec_verify_target_only needs (0 on invalid sizes). */
size_t spec_verify_target_only_workspace_size(int B, int K, int V, spec_dtype dtype);

/*
 * spec_verify_target_only — target-only verification of K greedy draft
 * tokens for B batch rows (Sec. 2.2, Eq. target_only).  The draft logits are
 * not read: the acceptance rule uses the target's probabilities only.
 *
 * For row b, with T = temperature[b] (or temperature_scalar):
 *   p_i = softmax(target[b, i, :] / T), i = 0..K (row K: bonus position)
 *   step i accepts x_i = draft_ids[b, i] (the draft's greedy token) iff u_i < p_i(x_i)
 *   n = first rejected step (K if none); accept_len[b] = n
 *   emitted[b, 0..n-1] = x_0..x_{n-1}; emitted[b, n+1..K] = -1
 *   emitted[b, n] = smallest v with C(v) > u' * Z, C the cumulative sum of
 *       r(v) = p_n(v) * 1[v != x_n] if n < K, else r = p_K; Z = sum r (if Z
 *       is 0 the sample is drawn from p_n).  The emitted token at position n
 *       is thereby distributed exactly as p_n.
 * Uniforms: the same Philox4x64-10 blocks as spec_verify (counter (b, i,
 *   offset, 0), key (seed, 0); word 0 accept test, word 1 resample).
 *
 * target_logits  [B, K+1, V] element strides (t_stride_b, t_stride_k), dtype
 * draft_ids      [B, K] int32, contiguous
 * temperature    [B] float32 device array, or NULL: temperature_scalar (finite, > 0)
 * accept_len     [B] int32 out; emitted_ids [B, K+1] int32 out, contiguous
 * p_at_draft     [B, K] float32 out: p_i(x_i) (may be NULL)
 * logz_target    [B, K+1] float32 out: natural-log partition function of z/T (may be NULL)
 * workspace      device memory of at least spec_verify_target_only_workspace_size bytes
 * Row data errors behave as in spec_verify (accept_len = -1, emitted = -1, NaN).
 * Limits: 1 <= K <= SPEC_MAX_K, 1 <= V <= SPEC_MAX_V, 1 <= B.
 */
spec_status spec_verify_target_only(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                                    spec_dtype dtype, int B, int K, int V,
                                    const int32_t* draft_ids,
                                    const float* temperature, float temperature_scalar,
                                    uint64_t seed, uint64_t offset,
                                    int32_t* accept_len, int32_t* emitted_ids,
                                    float* p_at_draft, float* logz_target,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spec_sample needs (0 on invalid sizes). */
size_t spec_sample_workspace_size(int R, int V, spec_dtype dtype);

/*
 * spec_sample — draft-stage token choice for R rows of logits (App. G.1, the
 * draft stage: temperature softmax and a multinomial draw).
 *
 * Row r with T = temperature[r] (or temperature_scalar):
 *   T > 0:  tokens[r] = smallest v with C(v) > u, C the cumulative sum of
 *           softmax(logits[r, :] / T), u = (word0 >> 40) * 2^-24 of
 *           Philox4x64-10(counter = (r, 0, offset, 1), key = (seed, 0))
 *           (counter word 3 = 1 keeps this stream apart from verification's);
 *           logz[r] = natural-log partition function of z/T
 *   T == 0: tokens[r] = the greedy token, the first index of the largest
 *           logit (the draft choice of spec_verify_target_only); logz[r] = NaN
 *
 * logits       [R, V], element stride stride_r between rows, dtype
 * temperature  [R] float32 device array, or NULL: temperature_scalar (finite, >= 0)
 * tokens       [R] int32 out
 * logz         [R] float32 out (may be NULL)
 * workspace    device memory of at least spec_sample_workspace_size bytes
 * Row data errors (NaN or +inf logits, all -inf, a per-row temperature that
 * is negative or not finite) give tokens[r] = -1 and logz[r] = NaN.
 * Limits: 1 <= R, 1 <= V <= SPEC_MAX_V.
 */
spec_status spec_sample(const void* logits, int64_t stride_r, spec_dtype dtype, int R, int V,
                        const float* temperature, float temperature_scalar,
                        uint64_t seed, uint64_t offset,
                        int32_t* tokens, float* logz,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Columns of the per-step output of spec_diagnostics. */
typedef enum SPEC_ENUM_INT {
  SPEC_DIAG_ENTROPY_TARGET = 0, /* H(p_i) in nats (Sec. 3.1)                               */
  SPEC_DIAG_ENTROPY_DRAFT = 1,  /* H(q_i) in nats                                           */
  SPEC_DIAG_MAX_P = 2,          /* max_v p_i(v) (Prop. to_entropy: >= exp(-H(p_i)))         */
  SPEC_DIAG_ALPHA_TO = 3,       /* p_i(argmax q_i), Eq. target_only                         */
  SPEC_DIAG_ALPHA_RS = 4,       /* sum_v min(p_i, q_i) = 1 - d_TV(p_i, q_i), Eq. reject_sample */
  SPEC_DIAG_ALPHA_P_GT_Q = 5,   /* sum over p > q of q                                      */
  SPEC_DIAG_ALPHA_Q_GE_P = 6,   /* sum over q >= p of p (columns 5 + 6 = column 4)          */
  SPEC_DIAG_NCOLS = 7
} spec_diag_column;

/* Bytes of workspace spec_diagnostics needs (0 on invalid sizes). */
size_t spec_diagnostics_workspace_size(int B, int K, int V, spec_dtype dtype);

/*
 * spec_diagnostics — per-step acceptance diagnostics (Sec. 3: target entropy
 * against acceptance; App. E: rejection sampling is preferred over
 * target-only verification iff d_TV(p, q) < 1 - p(argmax q)).
 *
 * For row b and step i < K, with T as in spec_verify, p_i = softmax(target[b, i] / T)
 * and q_i = softmax(draft[b, i] / T):
 *   diag[b, i, c] for the columns c of spec_diag_column;
 *   greedy_draft[b, i] = argmax_v q_i(v), first index among ties (may be NULL);
 *   rs_preferred[b, i] = 1 if alpha^RS > alpha^TO else 0 (may be NULL).
 * The split alpha_{p>q} / alpha_{q>=p} decides p > q per token in float32:
 * tokens whose p and q agree to about 1e-6 relative may land on either side.
 *
 * target_logits  [B, >= K, V] element strides (t_stride_b, t_stride_k); rows
 *                i < K are read, so a [B, K+1, V] verification tensor can be passed
 * draft_logits   [B, K, V] element strides (d_stride_b, d_stride_k)
 * temperature    [B] float32 device array, or NULL: temperature_scalar (finite, > 0)
 * diag           [B, K, SPEC_DIAG_NCOLS] float32 out, contiguous
 * workspace      device memory of at least spec_diagnostics_workspace_size bytes
 * Row data errors (as in spec_verify, without draft ids) give NaN in every
 * column, greedy_draft = -1 and rs_preferred = -1.
 * Limits: 1 <= K <= SPEC_MAX_K, 1 <= V <= SPEC_MAX_V, 1 <= B.
 */
spec_status spec_diagnostics(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                             const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                             spec_dtype dtype, int B, int K, int V,
                             const float* temperature, float temperature_scalar,
                             float* diag, int32_t* greedy_draft, int32_t* rs_preferred,
                             void* workspace, size_t workspace_bytes, void* stream);

typedef enum SPEC_ENUM_INT {
  SPEC_KL_FORWARD = 0, /* sum_v p_v log(p_v / q_v)   (App. B)                     */
  SPEC_KL_CE = 1,      /* -sum_v p_v log q_v        (= H(p) + forward KL)         */
  SPEC_KL_REVERSE = 2  /* sum_v q_v log(q_v / p_v)   (App. C)                     */
} spec_kl_kind;

/* Bytes of workspace spec_kl_loss_fwd_bwd needs (0 on invalid sizes). */
size_t spec_kl_workspace_size(int N, int K, int V, spec_dtype dtype);

/*
 * spec_kl_loss_fwd_bwd — the CE / forward-KL / reverse-KL objectives of the
 * draft against the (detached) target, the baselines of the TV loss (Sec.
 * 4.1 footnote, Table grad_comparison, App. B, App. C), and their gradients
 * w.r.t. the draft logits.
 *
 * For position n and draft step k, p = softmax(target[n, k] / T),
 * q = softmax(draft[n, k] / T), L_{n,k} by `kind` (terms with zero weight are 0):
 *   forward KL / CE:  grad = scale * (1/K) * (1/T) * (q - p)
 *   reverse KL:       grad = scale * (1/K) * (1/T) * q * (log q - log p - L_{n,k})
 *   loss = scale * sum_n (1/K) sum_k L_{n,k}
 * target_logits, draft_logits  [N, K, V], element strides (stride_n, stride_k)
 * temperature    finite and > 0
 * loss           [1] float32 out (device)
 * per_step       [N, K] float32 out: L_{n,k} (may be NULL)
 * grad_draft     [N, K, V] float32 out, contiguous; NULL = forward only
 * NaN or infinite logits propagate into that position's loss and gradient.
 * Limits: 1 <= K <= SPEC_MAX_K, 1 <= V <= SPEC_MAX_V, 1 <= N, N*K < 2^31.
 */
spec_status spec_kl_loss_fwd_bwd(const void* target_logits, int64_t t_stride_n, int64_t t_stride_k,
                                 const void* draft_logits, int64_t d_stride_n, int64_t d_stride_k,
                                 spec_dtype dtype, int N, int K, int V,
                                 float temperature, spec_kl_kind kind, float scale,
                                 float* loss, float* per_step, float* grad_draft,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* spec_status_string(spec_status s);

/* SPEC_VERSION of the built library. */
int spec_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECVERIFY_H */

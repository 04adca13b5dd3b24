// kl_kernel.h — CE, forward-KL and reverse-KL losses of the draft against the
// target and their gradients w.r.t. the draft logits (paper Sec. 4.1 and its
// footnote, Table grad_comparison, App. B, App. C): the objectives the TV
// loss is compared against.
//
//   1 kl_stats    every target and draft row, one wave per sub-chunk: the
//                 largest logit, how many elements hold it, and the sum of
//                 2^(z s - r) over every other element (r an integer
//                 reference), so that log2 of a normaliser dominated by one
//                 token is formed as log1p of a sum of small terms, not as
//                 the logarithm of a float32 sum near 1.
//   2 kl_norm     each row's log2 partition function in float64 and its
//                 per-element reference.
//     kl_top      reverse KL, per draft row: the target's logit at the
//                 row's first largest logit (a scan of the one sub-chunk
//                 that holds it).
//   3 kl_pass     per (position n, step k, chunk), with t = z_t s - M_t and
//                 u = z_d s - M_d (log2 units), e = 2^t, f = 2^u: Se = sum e,
//                 Sf = sum f and the weighted log-ratio sum W (forward:
//                 sum e (t - u); CE: sum e (-u)), all in float64 from the same
//                 e, f, t, u, so the loss (formed in kl_coef) is normalised by
//                 its own sums; for forward KL and CE, on the pairs whose
//                 largest probabilities nearly agree, also x = Z_d' - Z_t',
//                 the sum of 2^(b) - 2^(a) over every element, a and b its
//                 logits less each row's largest (times s), each term from
//                 the exact log ratio, and on the other pairs the gradient,
//                 written here; for reverse KL the sum of f (d - c),
//                 d = log2 q - log2 p and c its value at the draft's first
//                 largest logit, each d - c from exact logit differences.
//   4 kl_coef     per position: L_{n,k} from its chunks, the per-step output,
//                 the position loss, and the gradient constants: for forward
//                 KL and CE lam_t - lam_d = log2(Z_t' / Z_d') =
//                 log2(1 - x / Z_d'), for reverse KL mu - c.
//   5 kl_grad     the gradient, reading the pair again: every reverse-KL
//                 pair, and the forward-KL / CE pairs within the pair limit.
//   6 kl_loss     position losses added in a fixed order.
//
// Where p and q nearly agree, q - p and log q - log p are small differences
// of large terms.  Both are formed from d = log2 q - log2 p =
// ((z_d - z_t) - (zmax_d - zmax_t)) s + (lam_t - lam_d), lam = log2 Z - zmax s:
// the logits enter as exact differences (float64 for float32 logits, float32
// for bfloat16 logits, whose differences are exact there), and for forward
// KL and CE lam_t - lam_d comes from the pairwise sum x, not from two
// separately rounded partition functions, whose float32 error would set q - p
// of tokens that nearly coincide in the two rows (kl_needs_pairwise: only
// where the rows' largest probabilities lie within the pair limit).  Then
// q - p = sign(d) max(p, q) (1 - 2^-|d|), with 1 - 2^-x from its series
// below x = 1/2 and the difference of the two probabilities above.  For
// reverse KL the gradient q (d - mu) ln2 is invariant under a common shift of
// d (mu moves with it), so every log ratio is taken against c, its value at
// the draft's first largest logit: d - c = ((z_d - z_t) - (zmax_d - z_t at
// that logit)) s from exact logit differences, without the normalisers, and
// mu - c = sum_i q_i (d_i - c).  Where the draft's mass sits on tokens whose
// log ratios nearly agree, d - mu is then a difference of two small numbers
// rather than of two large ones.
#pragma once

#include <type_traits>

#include "sv_device.h"

namespace sv {

constexpr int kKlForward = 0;
constexpr int kKlCe = 1;
constexpr int kKlReverse = 2;

// Statistics of one sub-chunk of a row: its largest logit zmax, the number n
// of elements equal to it, and R = sum over the other elements of
// 2^(z s - r), r = ceil(zmax s) (an integer, so rescaling between
// references is exact).
struct KlStat {
  float zmax;
  int n;
  double R;
};

// A row's normaliser: p_v = 2^(z_v s - M) / D with M the integer reference.
// The log2 partition function is zmax s + lam; lam is kept apart because
// zmax s is large and its float64 rounding would swamp the log ratio of a
// token that holds nearly all the mass.
struct KlNorm {
  float M;
  float invD;
  float zmax;
  int n;
  double lam;  // log2(n + R 2^-(zmax s - M)) = log2 Z - zmax s
  double D;
  float zo;    // reverse KL, draft rows: the target's logit at the row's first largest logit (kl_top)
};

struct KlPart {  // one chunk of a (position, step) pair
  double se, sf, w;
  double x;  // forward KL / CE: Z_d' - Z_t', the sum of 2^(b) - 2^(a); reverse KL: sum f (d - c) (see kl_pass)
};

struct KlArgs {
  RowsDesc rows;  // target rows (n, k): tper = K; draft rows: dper = K
  int N, K, kind;
  double scale;
  float inv_t;
  float* loss; float* per_step; float* grad;
  KlStat* stats;         // [2 N K][SC]
  int SC;                // sub-chunks per row of the statistics pass
  KlNorm* norms;         // [2 N K]
  KlPart* parts;         // [N K][C]
  float4* coef;          // [N K]: reverse KL the gradient factor and mu - c; forward KL, CE lam_t - lam_d as hi + lo
  double pair_limit;     // forward KL, CE: |lam_t - lam_d| up to which x is summed pairwise
  double* loss_pos;      // [N]
  int vec_g;
};

// 2^(z s - r).  With CORR the exponent is carried beyond float32: z s = h + l
// exactly (h = z s rounded, l = fma(z, s, -h)), h - r is exact wherever h and
// the integer r are within a factor of two (the elements that carry the
// weight of the sum), and the dropped l enters to first order,
// 2^(h - r) (1 + l ln2).  Without CORR the exponent is fma(z, s, -r), rounded
// once.
template <bool CORR>
__device__ __forceinline__ float kl_term(float z, float s, float r) {
  if constexpr (CORR) {
    const float h = z * s;
    const float l = fmaf(z, s, -h);
    const float e = __builtin_amdgcn_exp2f(h - r);
    return e > 0.f ? fmaf(e * 0.69314718f, l, e) : e;  // 0, or NaN for a NaN logit
  } else {
    return __builtin_amdgcn_exp2f(fmaf(z, s, -r));
  }
}

// Statistics of every row at sub-chunk granularity, one wave per sub-chunk
// (ST tiles of 256 vectors, streamed S vectors per lane at a time).  Each
// lane keeps its largest logit, how often it occurred and the float64 sum of
// its other elements relative to its own reference; one wave maximum and
// float64 wave sums give the sub-chunk's record.
template <class E, int ST, int S, bool CORR>
__global__ __launch_bounds__(kThreads) void kl_stats_wave_kernel(RowsDesc d, int SC, KlStat* __restrict__ stats,
                                                                 int64_t nsub) {
  constexpr int EPV = E::EPV;
  constexpr int WV = ST * (kThreads / 64);
  static_assert(WV % S == 0, "whole load steps per sub-chunk");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kWaves + wave;
  if (g >= nsub) return;
  const int r = static_cast<int>(g / SC), j = static_cast<int>(g - static_cast<int64_t>(g / SC) * SC);
  int b;
  bool aligned;
  const typename E::raw* row = row_of<E>(d, r, &b, &aligned);
  const float s = scale_of(d.temp_scalar);
  const int e0 = j * WV * 64 * EPV;
  float zm = -INFINITY, rf = 0.f;
  int n = 0;
  double R = 0.0;
#pragma unroll 1
  for (int st = 0; st < WV / S; ++st) {
    const int es = e0 + st * S * 64 * EPV;
    if (es >= d.V) break;
    float x[S][EPV];
    load_span<E, S, 64>(row, es, lane, d.V, aligned, x);
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
      for (int k = 0; k < EPV; ++k) mx = fmaxf(mx, x[i][k]);
    if (mx > zm) {  // a new largest logit: the old one joins the other elements
      const float nr = ceilf(mx * s);
      if (zm != -INFINITY)
        R = ldexp(R, static_cast<int>(rf - nr)) + static_cast<double>(n) * static_cast<double>(kl_term<CORR>(zm, s, nr));
      zm = mx;
      rf = nr;
      n = 0;
    }
    if (zm != -INFINITY) {
#pragma unroll
      for (int i = 0; i < S; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float z = x[i][k];
          const float e = kl_term<CORR>(z, s, rf);
          const bool top = z == zm;
          n += top ? 1 : 0;
          acc += top ? 0.f : e;
        }
        R += static_cast<double>(acc);
      }
    }
  }
  const float zw = wave_max(zm);
  double Rl = 0.0;
  int nl = 0;
  if (zm == zw) {
    nl = n;
    Rl = R;
  } else if (zm != -INFINITY) {  // this lane's largest logit is one of the others
    const float rw = ceilf(zw * s);
    Rl = ldexp(R, static_cast<int>(rf - rw)) + static_cast<double>(n) * static_cast<double>(kl_term<CORR>(zm, s, rw));
  }
  if (R != R) Rl = R;  // NaN propagates (data error)
  Rl = wave_sum(Rl);
  double nd = wave_sum(static_cast<double>(nl));
  if (lane == 0) {
    KlStat o;
    o.zmax = zw;
    o.n = static_cast<int>(nd);
    o.R = Rl;
    stats[g] = o;
  }
}

// One wave per row: combine the row's SC sub-chunk records into its integer
// reference M, 1/D and lam = log2(n) + log1p(R / (n 2^(zmax s - M))) / ln 2,
// the log2 partition function less zmax s.
__global__ __launch_bounds__(kThreads) void kl_norm_kernel(const KlStat* __restrict__ stats, int rows, int SC,
                                                           float s, KlNorm* __restrict__ out) {
  const int r = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int lane = threadIdx.x & 63;
  const KlStat* st = stats + static_cast<int64_t>(r) * SC;
  float zm = -INFINITY;
  for (int c = lane; c < SC; c += 64) zm = fmaxf(zm, st[c].zmax);
  zm = wave_max(zm);
  const float rf = ceilf(zm * s);
  const double zs = static_cast<double>(zm) * static_cast<double>(s);  // exact
  double R = 0.0, nn = 0.0;
  bool nan = false;
  for (int c = lane; c < SC; c += 64) {
    const KlStat k = st[c];
    if (k.R != k.R) nan = true;
    if (k.zmax == -INFINITY) continue;
    if (k.zmax == zm) {
      nn += k.n;
      R += k.R;
    } else {
      const float rc = ceilf(k.zmax * s);
      R += ldexp(k.R, static_cast<int>(rc - rf)) +
           static_cast<double>(k.n) * exp2(static_cast<double>(k.zmax) * static_cast<double>(s) - rf);
    }
  }
  R = wave_sum(R);
  nn = wave_sum(nn);
  nan = __ballot(nan) != 0;
  if (lane == 0) {
    KlNorm o;
    o.M = rf;
    o.zmax = zm;
    o.n = static_cast<int>(nn);
    const double mt = exp2(zs - static_cast<double>(rf));
    o.D = nn * mt + R;
    o.lam = log2(nn) + log1p(R / (nn * mt)) * kLog2eD;
    if (nan) { o.D = NAN; o.lam = NAN; }
    o.invD = static_cast<float>(1.0 / o.D);
    o.zo = NAN;
    out[r] = o;
  }
}

// Reverse KL, one wave per (position, step): the target's logit at the
// draft row's first largest logit, into the draft row's norm.  The scan
// reads the first sub-chunk (SUB elements) whose statistics hold the row's
// largest logit.  Where no element matches (a row of NaN), the target's
// largest logit stands in: any finite reference gives the same gradient up
// to rounding.
template <class E, int SUB, int S>
__global__ __launch_bounds__(kThreads) void kl_top_kernel(RowsDesc d, const KlStat* __restrict__ stats, int SC,
                                                          KlNorm* __restrict__ norms, int NK) {
  constexpr int EPV = E::EPV;
  static_assert(SUB % (S * 64 * EPV) == 0, "whole load steps per sub-chunk");
  const int lane = threadIdx.x & 63;
  const int u = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (u >= NK) return;
  const float zm = norms[NK + u].zmax;
  const KlStat* st = stats + static_cast<int64_t>(NK + u) * SC;
  int c0 = SC;
  for (int c = lane; c < SC; c += 64)
    if (st[c].zmax == zm) c0 = min(c0, c);
  c0 = wave_min_int(c0);
  int idx = d.V;
  if (c0 < SC) {
    int b;
    bool al;
    const typename E::raw* rd = row_of<E>(d, NK + u, &b, &al);
    const int e0 = c0 * SUB, e1 = min(d.V, e0 + SUB);
    for (int es = e0; es < e1; es += S * 64 * EPV) {
      float x[S][EPV];
      load_span<E, S, 64>(rd, es, lane, d.V, al, x);
#pragma unroll
      for (int j = 0; j < S; ++j)
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const int e = es + j * 64 * EPV + lane * EPV + k;
          if (x[j][k] == zm && e < e1) idx = min(idx, e);
        }
    }
    idx = wave_min_int(idx);
  }
  if (lane == 0) {
    float zo = norms[u].zmax;
    if (idx < d.V) {
      int b;
      bool al;
      zo = E::one(row_of<E>(d, u, &b, &al) + idx);
    }
    norms[NK + u].zo = zo;
  }
}

// ((z_d - z_t) - (zmax_d - zmax_t)) s in float64 (log2 q - log2 p less lam_t - lam_d).
__device__ __forceinline__ double kl_wdiff(float zt, float zd, double c1, double s) {
  return ((static_cast<double>(zd) - static_cast<double>(zt)) - c1) * s;
}

// log2 q - log2 p of one element in float64,
// ((z_d - z_t) - (zmax_d - zmax_t)) s + (lam_t - lam_d): every logit
// difference is exact, and at the element holding both rows' largest logit
// only lam_t - lam_d remains, which carries no float32 sum near 1.
struct KlDelta {
  double c1;   // zmax_d - zmax_t
  double lam;  // lam_t - lam_d
  double s;
  float c1f, lam_hi, lam_lo, sf;  // the same in float32 (lam = lam_hi + lam_lo)
};
__device__ __forceinline__ void kl_delta_set_lam(KlDelta& r, double lam) {
  r.lam = lam;
  r.lam_hi = static_cast<float>(lam);
  r.lam_lo = static_cast<float>(lam - static_cast<double>(r.lam_hi));
}
__device__ __forceinline__ KlDelta kl_delta_ref(const KlNorm& t, const KlNorm& d, float s) {
  KlDelta r;
  r.c1 = static_cast<double>(d.zmax) - static_cast<double>(t.zmax);
  r.lam = t.lam - d.lam;
  r.s = static_cast<double>(s);
  r.c1f = static_cast<float>(r.c1);
  r.lam_hi = static_cast<float>(r.lam);
  r.lam_lo = static_cast<float>(r.lam - static_cast<double>(r.lam_hi));
  r.sf = s;
  return r;
}

// Reverse KL: d - c = ((z_d - z_t) - (zmax_d - zo)) s, zo the target's logit
// at the draft's first largest logit, as the wf of kl_ratio (no normalisers).
__device__ __forceinline__ KlDelta kl_delta_top(const KlNorm& d, float s) {
  KlDelta r;
  r.c1 = static_cast<double>(d.zmax) - static_cast<double>(d.zo);
  r.lam = 0.0;
  r.s = static_cast<double>(s);
  r.c1f = static_cast<float>(r.c1);
  r.lam_hi = 0.f;
  r.lam_lo = 0.f;
  r.sf = s;
  return r;
}

// The log ratios of one element: dl = log2 q - log2 p and wf = dl without
// the normaliser difference, ((z_d - z_t) - (zmax_d - zmax_t)) s.  Float32
// logits take them in float64.  For bfloat16 logits the logit differences
// are exact in float32 (or within one rounding when the two exponents lie
// more than 16 apart), so one float32 product and the normaliser
// difference in two floats leave an error of a few float32 roundings of
// |wf|, far inside the bfloat16 tolerance.
struct KlRatio {
  float dl, wf;
};
template <class E>
__device__ __forceinline__ KlRatio kl_ratio(float zt, float zd, const KlDelta& r) {
  KlRatio o;
  if constexpr (std::is_same<E, F32>::value) {
    const double wd = kl_wdiff(zt, zd, r.c1, r.s);
    o.dl = static_cast<float>(wd + r.lam);
    o.wf = static_cast<float>(wd);
  } else {
    const float w0 = (zd - zt) - r.c1f;
    o.wf = w0 * r.sf;
    o.dl = fmaf(w0, r.sf, r.lam_hi) + r.lam_lo;
  }
  return o;
}

// |q - p| of one element from its probabilities and the accurate log ratio:
// below |d| = 1/2 max(p, q) (1 - 2^-|d|) from the series (float32 logits:
// terms to y^7; bfloat16 logits: to y^4), above it max - min, whose
// rounding is then at most six times the two probabilities' own.
template <class E>
__device__ __forceinline__ float kl_absdiff(float mx, float mn, float d) {
  constexpr int D = std::is_same<E, F32>::value ? 6 : 3;
  const float ad = fabsf(d);
  return ad < 0.5f ? mx * one_minus_exp2_neg_small<D>(ad) : mx - mn;
}
__device__ __forceinline__ float kl_delta(float zt, float zd, const KlDelta& r) {
  return static_cast<float>(fma((static_cast<double>(zd) - static_cast<double>(zt)) - r.c1, r.s, r.lam));
}

// Forward KL / CE gradient of one element: sign(d) |q - p| scale / (K T)
// from e = 2^(z_t s - M_t), f = 2^(z_d s - M_d) and d = log2 q - log2 p.
template <class E>
__device__ __forceinline__ float kl_fwd_grad(float e, float f, float dl, const KlNorm& nt, const KlNorm& nd,
                                             float gcoef) {
  const float pe = e * nt.invD, qf = f * nd.invD;
  const float mx = fmaxf(pe, qf);
  const float g = kl_absdiff<E>(mx, fminf(pe, qf), dl);
  return mx > 0.f ? gcoef * copysignf(g, dl) : (mx == 0.f ? 0.f : mx);
}

// Write EPV gradient values of one vector (float4 stores when aligned).
template <int EPV>
__device__ __forceinline__ void store_grad(float* gr, int v0, int V, bool vec, const float (&gv)[EPV]) {
  if (vec && v0 + EPV <= V) {
#pragma unroll
    for (int h = 0; h < EPV; h += 4) {
      f32x4 w4 = {gv[h], gv[h + 1], gv[h + 2], gv[h + 3]};
      __builtin_nontemporal_store(w4, reinterpret_cast<f32x4*>(gr + v0 + h));
    }
  } else {
#pragma unroll
    for (int k = 0; k < EPV; ++k)
      if (v0 + k < V) gr[v0 + k] = gv[k];
  }
}

// Whether a (position, step) pair needs the pairwise x of kl_pass.  lam_t -
// lam_d = log2(max q / max p), so where it exceeds the limit the largest
// |q - p| of the row is at least (1 - 2^-limit) of the larger maximum, and the
// difference of the two separately summed normalisers (error a few 1e-7)
// moves no gradient element by more than that error over (1 - 2^-limit) of
// the row's largest (64 times it at the bfloat16 limit 1/64).  Both kl_pass
// and kl_coef take the decision from the same stored values.
__device__ __forceinline__ bool kl_needs_pairwise(const KlNorm& t, const KlNorm& d, double limit) {
  return fabs(t.lam - d.lam) <= limit;
}

// One task's sums for kl_pass: Σe, Σf, the weighted log-ratio sum and, by
// KIND, the reverse-KL sum of f (d - c) (dr: kl_delta_top) or, with X, the
// pairwise x.  With GW (forward KL / CE beyond the pair limit, dr carrying
// lam_t - lam_d of the two normalisers) the task also writes its gradient.
template <class E, int NT, int S, int KIND, bool X, bool GW>
__device__ __forceinline__ void kl_pass_sums(const typename E::raw* rt, bool al_t, const typename E::raw* rd,
                                             bool al_d, int tile0, int nt_tiles, int V, float s, const KlNorm& nt,
                                             const KlNorm& nd, const KlDelta& dr, double (&v)[4], float* gr,
                                             float gcoef, bool vec_g) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  double se = 0.0, sf = 0.0, w = 0.0, xs = 0.0;
  // 2^(z s - zmax s) = e 2^(M - zmax s): the scale of each row's elements against its largest
  float kt = 0.f, kd = 0.f;
  if (X) {
    kt = static_cast<float>(exp2(static_cast<double>(nt.M) - static_cast<double>(nt.zmax) * dr.s));
    kd = static_cast<float>(exp2(static_cast<double>(nd.M) - static_cast<double>(nd.zmax) * dr.s));
  }
#pragma unroll
  for (int j0 = 0; j0 < NT; j0 += S) {
    if (j0 >= nt_tiles) break;
    float xt[S][EPV], xd[S][EPV];
    load_tiles<E, S>(rt, tile0 + j0, V, al_t, xt);
    load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
    for (int j = 0; j < S; ++j) {
      // the EPV elements of one vector are summed in float32, vectors in float64
      float ve = 0.f, vf = 0.f, vw = 0.f, vx = 0.f;
      float gv[EPV];
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        const float tt = fmaf(xt[j][k], s, -nt.M);
        const float uu = fmaf(xd[j][k], s, -nd.M);
        const float e = __builtin_amdgcn_exp2f(tt);
        const float f = __builtin_amdgcn_exp2f(uu);
        if (GW) gv[k] = kl_fwd_grad<E>(e, f, kl_ratio<E>(xt[j][k], xd[j][k], dr).dl, nt, nd, gcoef);
        float term;
        if (KIND == kKlForward) term = e > 0.f ? e * (tt - uu) : 0.f;
        else if (KIND == kKlCe) term = e > 0.f ? -(e * uu) : 0.f;
        else term = 0.f;
        if (KIND == kKlReverse) {
          const float dc = kl_ratio<E>(xt[j][k], xd[j][k], dr).wf;
          vx += f > 0.f ? f * dc : 0.f;
        }
        ve += e;
        vf += f;
        vw += term;
        if (X) {
          // x = Z_d' - Z_t' from every element's 2^(b) - 2^(a), a and b its
          // logits less the rows' largest (Z' = sum 2^(.)), each formed
          // from the exact log ratio wf: kl_coef turns it into the log ratio
          // of the two partition functions that the gradient pass uses
          const float wf = kl_ratio<E>(xt[j][k], xd[j][k], dr).wf;
          const float ea = e * kt, fb = f * kd;
          const float mb = fmaxf(ea, fb);
          const float xv = kl_absdiff<E>(mb, fminf(ea, fb), wf);
          vx += mb > 0.f ? copysignf(xv, wf) : 0.f;
        }
      }
      se += static_cast<double>(ve);
      sf += static_cast<double>(vf);
      w += static_cast<double>(vw);
      if (KIND == kKlReverse || X) xs += static_cast<double>(vx);
      if (GW) store_grad<EPV>(gr, (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV, V, vec_g, gv);
    }
  }
  v[0] = se; v[1] = sf; v[2] = w; v[3] = xs;
}

// S tiles per load step with the pairwise x, SN without it.
template <class E, int NT, int S, int SN, int KIND>
__global__ __launch_bounds__(kThreads) void kl_pass_kernel(KlArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  __shared__ RedLds<4> red;
  const RowsDesc& d = a.rows;
  const int C = d.C, V = d.V, NK = a.N * a.K;
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, u, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, NK + u, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const KlNorm nt = a.norms[u], nd = a.norms[NK + u];
    const KlDelta dr = KIND == kKlReverse ? kl_delta_top(nd, s) : kl_delta_ref(nt, nd, s);
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, (V + TILE - 1) / TILE - tile0);
    double v[4];
    float* gr = a.grad ? a.grad + static_cast<int64_t>(u) * V : nullptr;
    const float gcoef = static_cast<float>(a.scale * static_cast<double>(a.inv_t) / a.K);
    // the same for the whole workgroup: one loop body runs.  Forward KL and
    // CE within the pair limit sum x (kl_grad writes their gradient later);
    // beyond it the gradient needs nothing but the two normalisers and is
    // written here, so kl_grad skips the pair.
    if (KIND != kKlReverse && kl_needs_pairwise(nt, nd, a.pair_limit))
      kl_pass_sums<E, NT, S, KIND, true, false>(rt, al_t, rd, al_d, tile0, nt_tiles, V, s, nt, nd, dr, v, gr, gcoef,
                                                a.vec_g != 0);
    else if (KIND != kKlReverse && gr)
      kl_pass_sums<E, NT, SN, KIND, false, true>(rt, al_t, rd, al_d, tile0, nt_tiles, V, s, nt, nd, dr, v, gr, gcoef,
                                                 a.vec_g != 0);
    else
      kl_pass_sums<E, NT, SN, KIND, false, false>(rt, al_t, rd, al_d, tile0, nt_tiles, V, s, nt, nd, dr, v, gr,
                                                  gcoef, a.vec_g != 0);
    wg_sum<4>(v, red);
    if (threadIdx.x == 0) {
      KlPart o;
      o.se = v[0]; o.sf = v[1]; o.w = v[2]; o.x = v[3];
      a.parts[t] = o;
    }
  }
}

// Per position (one wave each, 4 per workgroup): L_{n,k}, the per-step
// output, the position loss and the reverse-KL gradient constants.
__global__ __launch_bounds__(kThreads) void kl_coef_kernel(KlArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = blockIdx.x * kWaves + wave;
  if (n >= a.N) return;
  const int C = a.rows.C, K = a.K;
  double Ln = 0.0;
  for (int kk = 0; kk < K; ++kk) {
    double se = 0.0, sf = 0.0, w = 0.0;
    const KlPart* ps = a.parts + static_cast<int64_t>(n * K + kk) * C;
    for (int cc = lane; cc < C; cc += 64) {
      se += ps[cc].se; sf += ps[cc].sf; w += ps[cc].w;
    }
    se = wave_sum(se);
    sf = wave_sum(sf);
    w = wave_sum(w);
    double L;  // nats
    const KlNorm& nt = a.norms[static_cast<int64_t>(n) * K + kk];
    const KlNorm& nd = a.norms[static_cast<int64_t>(a.N) * K + static_cast<int64_t>(n) * K + kk];
    if (a.kind == kKlReverse) {
      double xc = 0.0;
      for (int cc = lane; cc < C; cc += 64) xc += ps[cc].x;
      xc = wave_sum(xc);
      // L = ln2 mu, mu = sum_j q_j d_j with q_j = f_j / Sf, taken as
      // c + (mu - c): c = d at the draft's first largest logit =
      // (zmax_t - zo) s + lam_t - lam_d, mu - c = sum_j f_j (d_j - c) / Sf
      const double mc = xc / sf;
      const double c = (static_cast<double>(nt.zmax) - static_cast<double>(nd.zo)) *
                           static_cast<double>(scale_of(a.rows.temp_scalar)) +
                       (nt.lam - nd.lam);
      L = kLn2D * (c + mc);
      if (lane == 0) {
        // gradient: scale/(K T) q ln2 ((d - c) - (mu - c))
        const double A = a.scale * static_cast<double>(a.inv_t) / K * kLn2D / sf;
        a.coef[static_cast<int64_t>(n) * K + kk] =
            make_float4(static_cast<float>(A), static_cast<float>(mc), 0.f, 0.f);
      }
    } else {
      const double le = log2(se), lf = log2(sf);
      L = (a.kind == kKlForward) ? w / se - le + lf : w / se + lf;
      L *= kLn2D;
      // the log ratio of the two partition functions, lam_t - lam_d =
      // log2(Z_t' / Z_d') = log2(1 - x / Z_d') with x = Z_d' - Z_t' summed
      // pairwise (Z' = 2^lam): not the difference of two separately rounded
      // sums, whose float32 error would set q - p of tokens that nearly
      // coincide in the two rows.  Where the two rows' largest probabilities
      // lie far enough apart that error is harmless, and neither pass forms x.
      double dlam = nt.lam - nd.lam;
      if (kl_needs_pairwise(nt, nd, a.pair_limit)) {  // the same for the whole wave
        double xs = 0.0;
        for (int cc = lane; cc < C; cc += 64) xs += ps[cc].x;
        xs = wave_sum(xs);
        const double r = -xs * exp2(-nd.lam);
        if (r > -1.0 && r < INFINITY && dlam - dlam == 0.0) dlam = log1p(r) * (1.0 / kLn2D);
      }
      if (lane == 0) {
        const float hi = static_cast<float>(dlam);
        a.coef[static_cast<int64_t>(n) * K + kk] =
            make_float4(hi, static_cast<float>(dlam - static_cast<double>(hi)), 0.f, 0.f);
      }
    }
    Ln += L;
    if (lane == 0 && a.per_step) a.per_step[static_cast<int64_t>(n) * K + kk] = static_cast<float>(L);
  }
  if (lane == 0) a.loss_pos[n] = a.scale * Ln / K;
}

// The gradient pass.  Forward KL and CE: (q - p) scale / (K T) =
// sign(d) |q - p| scale / (K T), d = log2 q - log2 p formed with the
// pairwise partition-function ratio of kl_coef.  Reverse KL: scale / (K T)
// q ln2 ((d - c) - (mu - c)).
template <class E, int NT, int S, int KIND>
__global__ __launch_bounds__(kThreads) void kl_grad_kernel(KlArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  // Forward KL / CE: one workgroup per (position, step) pair, its chunks in
  // turn, since every pair beyond the pair limit leaves at once; reverse
  // KL: one workgroup per chunk (ntasks of them).
  constexpr bool kPerPair = KIND != kKlReverse;
  const RowsDesc& d = a.rows;
  const int C = d.C, V = d.V, NK = a.N * a.K;
  const float gcoef = static_cast<float>(a.scale * static_cast<double>(a.inv_t) / a.K);
  const int64_t nitems = kPerPair ? static_cast<int64_t>(NK) : ntasks;
  for (int64_t it = blockIdx.x; it < nitems; it += gridDim.x) {
    const int u = kPerPair ? static_cast<int>(it) : static_cast<int>(it / C);
    const int c0 = kPerPair ? 0 : static_cast<int>(it - static_cast<int64_t>(u) * C);
    const int c1 = kPerPair ? C : c0 + 1;
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, u, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, NK + u, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const KlNorm nt = a.norms[u], nd = a.norms[NK + u];
    if (KIND != kKlReverse && !kl_needs_pairwise(nt, nd, a.pair_limit)) continue;  // written by kl_pass
    KlDelta dr = KIND == kKlReverse ? kl_delta_top(nd, s) : kl_delta_ref(nt, nd, s);
    const float4 A = a.coef[u];
    if (KIND != kKlReverse) kl_delta_set_lam(dr, static_cast<double>(A.x) + static_cast<double>(A.y));
    float* gr = a.grad + static_cast<int64_t>(u) * V;
    for (int c = c0; c < c1; ++c) {
      const int tile0 = c * NT;
      const int nt_tiles = min(NT, (V + TILE - 1) / TILE - tile0);
#pragma unroll
      for (int j0 = 0; j0 < NT; j0 += S) {
        if (j0 >= nt_tiles) break;
        float xt[S][EPV], xd[S][EPV];
        load_tiles<E, S>(rt, tile0 + j0, V, al_t, xt);
        load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
        for (int j = 0; j < S; ++j) {
          float gv[EPV];
#pragma unroll
          for (int k = 0; k < EPV; ++k) {
            const float f = __builtin_amdgcn_exp2f(fmaf(xd[j][k], s, -nd.M));
            const KlRatio rk = kl_ratio<E>(xt[j][k], xd[j][k], dr);
            if constexpr (KIND == kKlReverse) {
              const float tm = rk.wf - A.y;  // (d - c) - (mu - c)
              gv[k] = f > 0.f ? A.x * f * tm : (f == 0.f ? 0.f : f);
            } else {
              const float e = __builtin_amdgcn_exp2f(fmaf(xt[j][k], s, -nt.M));
              gv[k] = kl_fwd_grad<E>(e, f, rk.dl, nt, nd, gcoef);
            }
          }
          store_grad<EPV>(gr, (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV, V, a.vec_g != 0, gv);
        }
      }
    }
  }
}

// The total loss: position losses added in a fixed order by one workgroup.
__global__ __launch_bounds__(kThreads) void kl_loss_kernel(KlArgs a) {
  __shared__ RedLds<1> red;
  double acc = 0.0;
  for (int p = threadIdx.x; p < a.N; p += kThreads) acc += a.loss_pos[p];
  double v[1] = {acc};
  wg_sum<1>(v, red);
  if (threadIdx.x == 0) *a.loss = static_cast<float>(v[0]);
}

}  // namespace sv

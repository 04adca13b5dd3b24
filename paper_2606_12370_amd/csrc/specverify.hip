// specverify.hip — C ABI of libspecverify.so: argument validation, workspace
// layout and the launch sequences behind the entry points declared in
// include/specverify.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>
#include <cstddef>
#include <cstdint>
#include <type_traits>
#include <utility>

#include "specverify.h"
#include "sv_device.h"
#include "gumbel_kernel.h"
#include "kl_kernel.h"
#include "tv_kernel.h"
#include "variants_kernel.h"
#include "verify_kernel.h"
#include "fused_kernel.h"

namespace {

using sv::BF16;
using sv::F32;

// Chunk geometry: a chunk is NT tiles of one 16-byte vector per thread,
// 16384 elements for both dtypes, read S tiles per step.
constexpr int kNtBf16 = 8;
constexpr int kNtF32 = 16;
constexpr int kStep = 4;
// Multinomial verification, target-only verification, the sampler and the
// diagnostics keep statistics per sub-chunk of kStep tiles (8192 bf16 or 4096
// fp32 elements), which is what their per-row launches read again; one wave
// streams one sub-chunk, kStatVec (statistics), kPairVec (verification pair
// pass), kDiagStatVec / kDiagPairVec (diagnostics) vectors per lane at a time.
constexpr int kStatVec = 8;
// (2 vectors per load step in the wave-stride pair pass: B=256, K=3,
// V=151936 bf16 177.6 against 179.0 us per call with 4, K=1 88.0 against
// 90.8; B=1024, V=262144 1074 against 1068)
constexpr int kPairVec = 2;
// Pair-pass items below which a launch of residual-step items only gives
// each one a workgroup (the small-batch launch shape).
constexpr int64_t kSharedItems = 8192;
// Residual-step items up to which the pair pass takes them first (about the
// waves the device holds at once).
constexpr int64_t kLongestFirstItems = 8192;
constexpr int kDiagPairVec = 2;
// (4 vectors per load step for the diagnostics statistics: 166.5-167.5
// against 170.1-170.6 us per call with 8 at B=256, K=3, V=151936 bf16)
constexpr int kDiagStatVec = 4;
constexpr int kChunkElems = 16384;
static_assert(kNtBf16 * sv::kThreads * sv::BF16::EPV == kChunkElems, "chunk geometry");
static_assert(kNtF32 * sv::kThreads * sv::F32::EPV == kChunkElems, "chunk geometry");
static_assert(kChunkElems % (sv::kThreads * sv::BF16H::EPV) == 0, "chunk geometry");
static_assert(sv::kDiagCols == SPEC_DIAG_NCOLS, "diagnostics columns");

template <class E> struct GradElem { using type = E; };
template <> struct GradElem<sv::BF16> { using type = sv::BF16H; };

int epv_of(spec_dtype dt) { return dt == SPEC_BF16 ? BF16::EPV : F32::EPV; }
int nt_of(spec_dtype dt) { return dt == SPEC_BF16 ? kNtBf16 : kNtF32; }
size_t esize_of(spec_dtype dt) { return dt == SPEC_BF16 ? 2 : 4; }
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Geometry {
  int ntiles = 0;  // tiles per row
  int C = 0;       // chunks per row
};

Geometry geometry(int V, spec_dtype dt) {
  Geometry g;
  const int64_t tile = static_cast<int64_t>(sv::kThreads) * epv_of(dt);
  g.ntiles = static_cast<int>((V + tile - 1) / tile);
  g.C = (g.ntiles + nt_of(dt) - 1) / nt_of(dt);
  return g;
}

// Sub-chunks of kStep tiles per row (the statistics granularity of multinomial verification).
int sub_chunks(int V, spec_dtype dt) { return (geometry(V, dt).ntiles + kStep - 1) / kStep; }

// Slices of kSliceTiles tiles per row: the granularity of the single-read
// verification (one workgroup per slice, two vectors per thread and row).
constexpr int kSliceTiles = 2;
static_assert(kSliceTiles == sv::kFusedNV, "a slice is one vector per thread per tile");
int slices(int V, spec_dtype dt) { return (geometry(V, dt).ntiles + kSliceTiles - 1) / kSliceTiles; }

// Largest vocabulary: element indices are 32-bit and run up to one chunk
// (16384 elements) past V where a row's last chunk is rounded up.
constexpr int64_t kMaxV = SPEC_MAX_V;
static_assert(kMaxV + kChunkElems < (int64_t{1} << 31), "element indices fit in int");

bool verify_sizes_ok(int B, int K, int V, spec_dtype dt) {
  if (B < 1 || K < 1 || K > SPEC_MAX_K || V < 1 || V > kMaxV) return false;
  const int64_t rows = static_cast<int64_t>(B) * (2 * K + 1);
  return rows * sub_chunks(V, dt) < (int64_t{1} << 31);
}

bool tv_sizes_ok(int N, int K, int V, spec_dtype dt) {
  if (N < 1 || K < 1 || K > SPEC_MAX_K || V < 1 || V > kMaxV) return false;
  const int64_t rows = static_cast<int64_t>(N) * 2 * K;
  return rows * std::max(geometry(V, dt).C, sub_chunks(V, dt)) < (int64_t{1} << 31);
}

bool rows_ok(int64_t rows, int V, spec_dtype dt) {
  return rows >= 1 && V >= 1 && V <= kMaxV && rows * geometry(V, dt).C < (int64_t{1} << 31);
}

// Sizes for the entry points that keep statistics per sub-chunk of kStep tiles.
bool rows_sub_ok(int64_t rows, int V, spec_dtype dt) {
  return rows >= 1 && V >= 1 && V <= kMaxV && rows * sub_chunks(V, dt) < (int64_t{1} << 31);
}

struct VerifyLayout {
  size_t stats = 0, norms = 0, decision = 0, pairs = 0, gbest = 0, total = 0;
};
VerifyLayout verify_layout(int B, int K, int V, spec_dtype dt, bool gumbel = false) {
  VerifyLayout L;
  // multinomial verification: room for the per-slice records of the single-read path
  // (two per sub-chunk of the chain)
  const size_t C = static_cast<size_t>(gumbel ? geometry(V, dt).C : slices(V, dt));
  // Gumbel-max verification keeps its statistics per sub-chunk, the rest per chunk
  const size_t CS = gumbel ? std::max(C, static_cast<size_t>(sub_chunks(V, dt))) : C;
  const size_t rows = static_cast<size_t>(B) * (2 * K + 1);
  size_t off = 0;
  L.stats = off; off = align_up(off + rows * CS * sizeof(sv::RowStat), 256);
  L.norms = off; off = align_up(off + rows * sizeof(sv::RowNorm), 256);
  L.decision = off; off = align_up(off + static_cast<size_t>(B) * sizeof(int32_t), 256);
  L.pairs = off; off = align_up(off + static_cast<size_t>(B) * K * C * sizeof(sv::PairStat), 256);
  if (gumbel) {  // per (batch row, chunk) best Gumbel keys
    L.gbest = off; off = align_up(off + static_cast<size_t>(B) * C * sizeof(sv::GumbelBest), 256);
  }
  L.total = off;
  return L;
}

struct TvLayout {
  size_t stats = 0, norms = 0, pairs = 0, coef = 0, loss = 0, bits = 0, bits_stride = 0, total = 0;
};
TvLayout tv_layout(int N, int K, int V, spec_dtype dt) {
  TvLayout L;
  const size_t C = static_cast<size_t>(geometry(V, dt).C);
  // statistics per sub-chunk of kStep tiles, the rest per chunk
  const size_t CS = std::max(C, static_cast<size_t>(sub_chunks(V, dt)));
  const size_t rows = static_cast<size_t>(N) * 2 * K;
  size_t off = 0;
  L.stats = off; off = align_up(off + rows * CS * sizeof(sv::RowStat), 256);
  L.norms = off; off = align_up(off + rows * sizeof(sv::RowNorm), 256);
  L.pairs = off; off = align_up(off + static_cast<size_t>(N) * K * C * sizeof(sv::TvPair), 256);
  L.coef = off; off = align_up(off + static_cast<size_t>(N) * K * sizeof(float2), 256);
  L.loss = off; off = align_up(off + static_cast<size_t>(N) * sizeof(double), 256);
  // indicator bits 1[q <= p] for the gradient pass: one 64-bit word per thread and chunk
  L.bits_stride = C * sv::kChunkWords * sizeof(uint64_t);
  L.bits = off; off = align_up(off + static_cast<size_t>(N) * K * L.bits_stride, 256);
  L.total = off;
  return L;
}

struct KlLayout {
  size_t stats = 0, norms = 0, parts = 0, coef = 0, loss = 0, total = 0;
};
KlLayout kl_layout(int N, int K, int V, spec_dtype dt) {
  KlLayout L;
  const size_t C = static_cast<size_t>(geometry(V, dt).C);
  const size_t SC = static_cast<size_t>(sub_chunks(V, dt));
  const size_t rows = static_cast<size_t>(N) * 2 * K;
  size_t off = 0;
  L.stats = off; off = align_up(off + rows * SC * sizeof(sv::KlStat), 256);
  L.norms = off; off = align_up(off + rows * sizeof(sv::KlNorm), 256);
  L.parts = off; off = align_up(off + static_cast<size_t>(N) * K * C * sizeof(sv::KlPart), 256);
  L.coef = off; off = align_up(off + static_cast<size_t>(N) * K * sizeof(float4), 256);
  L.loss = off; off = align_up(off + static_cast<size_t>(N) * sizeof(double), 256);
  L.total = off;
  return L;
}

struct ToLayout {
  size_t stats = 0, total = 0;
};
ToLayout to_layout(int B, int K, int V, spec_dtype dt) {
  ToLayout L;
  const size_t C = static_cast<size_t>(sub_chunks(V, dt));
  L.stats = 0;
  L.total = align_up(static_cast<size_t>(B) * (K + 1) * C * sizeof(sv::RowStat), 256);
  return L;
}

size_t sample_ws(int R, int V, spec_dtype dt) {
  return align_up(static_cast<size_t>(R) * sub_chunks(V, dt) * sizeof(sv::RowStat), 256);
}

struct DiagLayout {
  size_t stats = 0, norms = 0, info = 0, pairs = 0, total = 0;
};
DiagLayout diag_layout(int B, int K, int V, spec_dtype dt) {
  DiagLayout L;
  const size_t C = static_cast<size_t>(sub_chunks(V, dt));
  const size_t rows = static_cast<size_t>(B) * 2 * K;
  size_t off = 0;
  L.stats = off; off = align_up(off + rows * C * sizeof(sv::DiagStat), 256);
  L.norms = off; off = align_up(off + rows * sizeof(sv::RowNorm), 256);
  L.info = off; off = align_up(off + rows * sizeof(sv::DiagRow), 256);
  L.pairs = off; off = align_up(off + static_cast<size_t>(B) * K * C * sizeof(sv::DiagPair), 256);
  L.total = off;
  return L;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
// Both strides keep 16-byte vectors aligned (the products are taken modulo
// 2^64, which leaves them unchanged modulo 16).
bool rows_vec_aligned(const void* base, int64_t s0, int64_t s1, size_t esize) {
  return aligned16(base) && (static_cast<uint64_t>(s0) * esize) % 16 == 0 &&
         (static_cast<uint64_t>(s1) * esize) % 16 == 0;
}

// The last byte a tensor of n0 x n1 rows of V elements (strides s0, s1 in
// elements, both >= 0) occupies from base lies within the address space: the
// kernels' 64-bit row offsets then never overflow.
bool extent_ok(const void* base, int64_t n0, int64_t s0, int64_t n1, int64_t s1, int V, size_t esize) {
  int64_t a, b, last, bytes;
  if (__builtin_mul_overflow(n0 - 1, s0, &a) || __builtin_mul_overflow(n1 - 1, s1, &b) ||
      __builtin_add_overflow(a, b, &last) || __builtin_add_overflow(last, static_cast<int64_t>(V), &last) ||
      __builtin_mul_overflow(last, static_cast<int64_t>(esize), &bytes))
    return false;
  uintptr_t end;
  return !__builtin_add_overflow(reinterpret_cast<uintptr_t>(base), static_cast<uintptr_t>(bytes), &end);
}

// Statistics per sub-chunk of every row, one wave per sub-chunk and four
// waves per workgroup (one workgroup per four sub-chunks measured faster
// than a resident grid for this purely streaming pass).
template <class E>
void launch_stats_wave(const sv::RowsDesc& d, sv::RowStat* stats, int64_t rows, hipStream_t s) {
  const int64_t nsub = rows * d.C;
  hipLaunchKernelGGL((sv::row_stats_wave_kernel<E, kStep, kStatVec>),
                     dim3(static_cast<unsigned>((nsub + sv::kWaves - 1) / sv::kWaves)), dim3(sv::kThreads), 0, s, d,
                     stats, nsub);
}

// ---- single-read verification: launch facts per device ----------------------
// Resident workgroups per CU of each instantiation of the single-read kernel
// (dtype x K), the CU count and cooperative-launch support, queried once per
// device and read-only afterwards.
constexpr int kFusedMaxK = 4;
constexpr int kMaxDevices = 64;
struct FusedFacts {
  std::atomic<int> ready{0};
  int cus = 0, coop = 0;
  int bpc[2][kFusedMaxK + 1] = {};
};
FusedFacts g_fused_facts[kMaxDevices];
std::mutex g_fused_mu;

template <class E, int K>
const void* fused_kernel_ptr() {
  return reinterpret_cast<const void*>(&sv::verify_fused_kernel<E, K>);
}
template <class E>
const void* fused_kernel_for(int K) {
  switch (K) {
    case 1: return fused_kernel_ptr<E, 1>();
    case 2: return fused_kernel_ptr<E, 2>();
    case 3: return fused_kernel_ptr<E, 3>();
    case 4: return fused_kernel_ptr<E, 4>();
  }
  return nullptr;
}

const FusedFacts* fused_facts() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  FusedFacts& f = g_fused_facts[dev];
  if (f.ready.load(std::memory_order_acquire)) return &f;
  std::lock_guard<std::mutex> lk(g_fused_mu);
  if (!f.ready.load(std::memory_order_relaxed)) {
    int cus = 0, coop = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess) coop = 0;
    f.cus = cus;
    f.coop = coop;
    for (int k = 1; k <= kFusedMaxK; ++k) {
      int nb = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fused_kernel_for<BF16>(k), sv::kThreads, 0) != hipSuccess)
        nb = 0;
      f.bpc[SPEC_BF16][k] = nb;
      nb = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fused_kernel_for<F32>(k), sv::kThreads, 0) != hipSuccess)
        nb = 0;
      f.bpc[SPEC_F32][k] = nb;
    }
    (void)hipGetLastError();
    f.ready.store(1, std::memory_order_release);
  }
  return &f;
}

// Workgroups of the single-read kernel the device holds at once, or 0 when the
// shape does not qualify: K <= 4, 16-byte aligned rows whose length is a
// multiple of the 16-byte vector (8 bf16 or 4 fp32 elements), at most 64
// slices per row (the combine is one wave), cooperative launch, and room for
// at least one group of G = slices workgroups.
int fused_capacity(const sv::VerifyArgs& a, spec_dtype dt) {
  const int G = slices(a.rows.V, dt);
  const int epv = dt == SPEC_BF16 ? sv::BF16::EPV : sv::F32::EPV;
  if (a.K < 1 || a.K > kFusedMaxK || !a.rows.vec_t || !a.rows.vec_d || G > 64 || a.rows.V % epv != 0) return 0;
  const FusedFacts* f = fused_facts();
  if (!f || !f->coop || f->cus <= 0) return 0;
  const int cap = f->bpc[dt][a.K] * f->cus;
  return cap >= G ? cap : 0;
}

// Number of groups: as many as the device holds at once, at most one per
// batch row.
int fused_groups(int B, int G, int cap) { return std::min(cap / G, B); }

template <class E>
spec_status launch_verify_fused(sv::VerifyArgs a, int groups, hipStream_t s) {
  // statistics, overlaps and residual sums per slice; the finish inverts the
  // CDF inside one slice
  const int G = a.rows.C = slices(a.rows.V, std::is_same<E, BF16>::value ? SPEC_BF16 : SPEC_F32);
  // the record array starts all ones: a record is complete once it is not
  const int64_t words = int64_t{a.B} * (2 * a.K + 1) * G * 2;
  hipLaunchKernelGGL(sv::fill_ones_kernel, dim3(static_cast<unsigned>(std::min<int64_t>((words + 255) / 256, 1024))),
                     dim3(sv::kThreads), 0, s, reinterpret_cast<uint64_t*>(const_cast<sv::RowStat*>(a.stats)), words);
  int Gv = G, NG = groups;
  // about a second of polling before a wait gives up (never reached while the
  // cooperative launch keeps every workgroup resident)
  unsigned spin_limit = 1u << 20;
  void* args[] = {&a, &Gv, &NG, &spin_limit};
  if (hipLaunchCooperativeKernel(fused_kernel_for<E>(a.K), dim3(static_cast<unsigned>(G * NG)), dim3(sv::kThreads),
                                 args, 0, s) != hipSuccess)
    return SPEC_EHIP;
  hipLaunchKernelGGL((sv::finish_kernel<E, kSliceTiles, kSliceTiles>), dim3(static_cast<unsigned>(a.B)),
                     dim3(sv::kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E>
spec_status launch_verify(const sv::VerifyArgs& a, int64_t rows, hipStream_t s, const spec_launch* lc = nullptr) {
  const spec_dtype dt = std::is_same<E, BF16>::value ? SPEC_BF16 : SPEC_F32;
  // the automatic choice is the chain: on MI355X it measures faster than the
  // single-read path at every benchmarked shape (B = 64..1024, K = 3, bf16)
  const int path = lc ? lc->path : SPEC_PATH_AUTO;
  if (path == SPEC_PATH_SINGLE_READ) {
    const int cap = fused_capacity(a, dt);
    const int G = slices(a.rows.V, dt);
    int groups = cap ? fused_groups(a.B, G, cap) : 0;
    if (lc && lc->groups > 0) groups = (cap && lc->groups <= std::min(cap / G, a.B)) ? lc->groups : 0;
    if (groups > 0) return launch_verify_fused<E>(a, groups, s);
    return SPEC_EUNSUPPORTED;
  }
  // statistics and pair sums per sub-chunk of kStep tiles, one wave per sub-chunk
  launch_stats_wave<E>(a.rows, const_cast<sv::RowStat*>(a.stats), rows, s);
  hipLaunchKernelGGL((sv::decide_kernel<E>), dim3(static_cast<unsigned>(a.B)), dim3(sv::kThreads), 0, s, a);
  // pair pass: without overlaps only each batch row's residual step is read
  // again.  One wave per item, four per workgroup (measured faster than a
  // grid of what the device holds at once striding over them), or one
  // workgroup per item for launches whose every item is a residual-step item
  // (calls without overlaps, and K = 1) with fewer than kSharedItems items.
  // Measured with warm clocks, the two shapes interleaved (K = 3, V = 151936
  // bf16 unless noted; us per call): without overlaps B = 64 54.8 against
  // 64.5, B = 256 136.4 against 137.6, B = 512 247.3 against 245.6, B = 1024
  // 474.1 against 461.0; K = 1 B = 256 95.4 against 101.0, B = 512 163.7
  // against 161.6, B = 1024 302.2 against 285.0; with overlaps at K = 3 the
  // wave shape is faster at every B measured (64: 70.2 against 71.5, 128:
  // 106.5 against 114.3, 256: 183.2 against 200.3)
  const int64_t items = int64_t{a.B} * (a.overlap ? a.K : 1) * a.rows.C;
  const int shape = lc ? lc->residual_shape : 0;
  const bool residual_only = a.overlap == nullptr || a.K == 1;
  const int split = shape == 2 || (shape == 0 && residual_only && items < kSharedItems) ? 1 : 0;
  const int64_t wgs = split ? items : (items + sv::kWaves - 1) / sv::kWaves;
  // residual-step items first while they fit in about one round of what the
  // device holds at once, else the pair order (without overlaps every item
  // is a residual-step item)
  const int longest_first = (a.overlap == nullptr || int64_t{a.B} * a.rows.C <= kLongestFirstItems) ? 1 : 0;
  hipLaunchKernelGGL((sv::pair_pass_wave_kernel<E, kStep, kPairVec>), dim3(static_cast<unsigned>(wgs)),
                     dim3(sv::kThreads), 0, s, a, items, split, longest_first);
  // the finish inverts the CDF inside one sub-chunk (kStep tiles, one load step)
  hipLaunchKernelGGL((sv::finish_kernel<E, kStep, kStep>), dim3(static_cast<unsigned>(a.B)), dim3(sv::kThreads), 0,
                     s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E, int NT>
spec_status launch_verify_gumbel(const sv::VerifyArgs& a, sv::GumbelBest* gbest, int64_t rows, hipStream_t s) {
  const int C = a.rows.C;
  // the statistics per sub-chunk of kStep tiles with the chain's wave-shaped
  // pass (6.6 against 6.3 TB/s for the one-workgroup-per-chunk one), and the
  // decision combining them; the overlap and Gumbel passes keep their chunks
  sv::VerifyArgs as = a;
  as.rows.C = sub_chunks(a.rows.V, std::is_same<E, BF16>::value ? SPEC_BF16 : SPEC_F32);
  launch_stats_wave<E>(as.rows, const_cast<sv::RowStat*>(a.stats), rows, s);
  hipLaunchKernelGGL((sv::decide_kernel<E>), dim3(static_cast<unsigned>(a.B)), dim3(sv::kThreads), 0, s, as);
  if (a.overlap) {  // overlaps only: the Gumbel pass needs no residual mass
    void (*pp)(sv::VerifyArgs, int64_t) = sv::pair_pass_kernel<E, NT, kStep>;
    const int64_t pairs = int64_t{a.B} * a.K * C;
    hipLaunchKernelGGL(pp, dim3(static_cast<unsigned>(pairs)), dim3(sv::kThreads), 0, s, a,
                       pairs);
  }
  void (*gp)(sv::VerifyArgs, sv::GumbelBest*, int64_t) = sv::gumbel_pass_kernel<E, NT, kStep>;
  const int64_t tasks = int64_t{a.B} * C;
  hipLaunchKernelGGL(gp, dim3(static_cast<unsigned>(tasks)), dim3(sv::kThreads), 0, s, a,
                     gbest, tasks);
  hipLaunchKernelGGL(sv::gumbel_finish_kernel, dim3(static_cast<unsigned>((a.B + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a, static_cast<const sv::GumbelBest*>(gbest));
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E, int NT>
spec_status launch_sample_gumbel(const sv::GumbelSampleArgs& a, hipStream_t s) {
  const int64_t tasks = int64_t{a.R} * a.rows.C;
  // two tiles per load step (153.5-153.9 against 160.9-161.3 us per call for
  // 768 rows of V=151936 bf16)
  void (*gp)(sv::GumbelSampleArgs, int64_t) = sv::gumbel_sample_pass_kernel<E, NT, 2>;
  hipLaunchKernelGGL(gp, dim3(static_cast<unsigned>(tasks)), dim3(sv::kThreads), 0, s, a, tasks);
  hipLaunchKernelGGL(sv::gumbel_sample_finish_kernel, dim3(static_cast<unsigned>((a.R + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E, int NT>
spec_status launch_tv(const sv::TvArgs& a, hipStream_t s) {
  const int64_t units = int64_t{a.N} * a.K;
  const int C = a.rows.C;
  // the statistics per sub-chunk of kStep tiles with the wave-shaped pass,
  // and the normalisers combining them; the pair and gradient passes keep
  // their chunks
  sv::RowsDesc ds = a.rows;
  ds.C = sub_chunks(a.rows.V, std::is_same<E, BF16>::value ? SPEC_BF16 : SPEC_F32);
  launch_stats_wave<E>(ds, const_cast<sv::RowStat*>(a.stats), 2 * units, s);
  hipLaunchKernelGGL(sv::row_norm_kernel, dim3(static_cast<unsigned>((2 * units + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a.stats, static_cast<int>(2 * units), ds.C,
                     const_cast<sv::RowNorm*>(a.norms));
  void (*tp)(sv::TvArgs, int64_t) = sv::tv_pair_kernel<E, NT, kStep>;
  // one workgroup per task (measured faster than a resident grid: 5.6 against 6.0 ms at N=16384, K=3, V=151936)
  hipLaunchKernelGGL(tp, dim3(static_cast<unsigned>(units * C)), dim3(sv::kThreads), 0, s, a, units * C);
  hipLaunchKernelGGL(sv::tv_coef_kernel, dim3(static_cast<unsigned>((a.N + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a);
  // the gradient pass reads bf16 as 4-element vectors: one coalesced float4 store per lane
  using G = typename GradElem<E>::type;
  if (a.grad) {
    void (*tg)(sv::TvArgs, int64_t) = sv::tv_grad_kernel<G, kChunkElems / (sv::kThreads * G::EPV), kStep, E::EPV>;
    // one workgroup per task (measured faster than a resident grid for this read+write pass)
    hipLaunchKernelGGL(tg, dim3(static_cast<unsigned>(units * C)), dim3(sv::kThreads), 0, s, a, units * C);
  }
  hipLaunchKernelGGL(sv::tv_loss_kernel, dim3(1), dim3(sv::kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E, int NT, int KIND>
spec_status launch_kl(const sv::KlArgs& a, hipStream_t s) {
  const int64_t units = int64_t{a.N} * a.K;
  const int C = a.rows.C;
  // statistics per sub-chunk, one wave each; float32 logits carry their
  // exponents beyond float32 (their tolerance is 200 times tighter)
  const int64_t nsub = 2 * units * a.SC;
  constexpr bool kCorr = std::is_same<E, sv::F32>::value;
  hipLaunchKernelGGL((sv::kl_stats_wave_kernel<E, kStep, kStatVec, kCorr>),
                     dim3(static_cast<unsigned>((nsub + sv::kWaves - 1) / sv::kWaves)), dim3(sv::kThreads), 0, s,
                     a.rows, a.SC, a.stats, nsub);
  hipLaunchKernelGGL(sv::kl_norm_kernel, dim3(static_cast<unsigned>((2 * units + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, static_cast<const sv::KlStat*>(a.stats), static_cast<int>(2 * units),
                     a.SC, sv::scale_of(a.rows.temp_scalar), a.norms);
  if (KIND == sv::kKlReverse) {
    // the reference logit of the reverse-KL log ratios (one sub-chunk read per draft row)
    constexpr int kSub = kStep * sv::kThreads * E::EPV;
    hipLaunchKernelGGL((sv::kl_top_kernel<E, kSub, 4>), dim3(static_cast<unsigned>((units + sv::kWaves - 1) / sv::kWaves)),
                       dim3(sv::kThreads), 0, s, a.rows, static_cast<const sv::KlStat*>(a.stats), a.SC, a.norms,
                       static_cast<int>(units));
  }
  // the gradient pass reads bf16 as 4-element vectors, so that each lane
  // writes one float4; so does the forward-KL / CE statistics pass (with
  // 16-byte vectors it needs 124 VGPRs and measured 11.0 against 9.8 ms at
  // N=16384, K=3, V=151936), while the reverse-KL one reads 16-byte vectors
  // (6.8 against 7.2 ms)
  using G = typename GradElem<E>::type;
  using P = typename std::conditional<KIND == sv::kKlReverse, E, G>::type;
  constexpr int NTP = kChunkElems / (sv::kThreads * P::EPV);
  constexpr int NTG = kChunkElems / (sv::kThreads * G::EPV);
  // tiles per load step: 2 for the forward-KL / CE pass with the pairwise x
  // (24.5-24.8 against 25.6-25.8 ms per call), 4 for its loop body without
  // x (forward KL 21.2-21.4 against 22.4-22.7 ms; 8: 21.0-21.4), 2 for the
  // reverse-KL pass (21.1-21.2 against 21.3-21.7 ms with 4, 22.5 with 8)
  constexpr int SP = 2;
  constexpr int SPN = KIND == sv::kKlReverse ? 2 : kStep;
  void (*kp)(sv::KlArgs, int64_t) = sv::kl_pass_kernel<P, NTP, SP, SPN, KIND>;
  // one workgroup per task (measured faster than a resident grid: reverse KL 22.8 -> 21.2 ms per call)
  hipLaunchKernelGGL(kp, dim3(static_cast<unsigned>(units * C)), dim3(sv::kThreads), 0, s, a,
                     units * C);
  hipLaunchKernelGGL(sv::kl_coef_kernel, dim3(static_cast<unsigned>((a.N + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a);
  if (a.grad) {
    // reverse KL: one workgroup per chunk; forward KL / CE: one per pair (only
    // the pairs within the pair limit are left to write)
    void (*kg)(sv::KlArgs, int64_t) = sv::kl_grad_kernel<G, NTG, kStep, KIND>;
    const int64_t grid = KIND == sv::kKlReverse ? units * C : units;
    hipLaunchKernelGGL(kg, dim3(static_cast<unsigned>(grid)), dim3(sv::kThreads), 0, s, a, units * C);
  }
  hipLaunchKernelGGL(sv::kl_loss_kernel, dim3(1), dim3(sv::kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E, int NT>
spec_status launch_kl_kind(const sv::KlArgs& a, hipStream_t s) {
  if (a.kind == sv::kKlForward) return launch_kl<E, NT, sv::kKlForward>(a, s);
  if (a.kind == sv::kKlCe) return launch_kl<E, NT, sv::kKlCe>(a, s);
  return launch_kl<E, NT, sv::kKlReverse>(a, s);
}

// Target-only verification and the sampler keep statistics per sub-chunk
// of kStep tiles (as multinomial verification does), so that their per-row
// launch reads one sub-chunk again, in one load step.
template <class E>
spec_status launch_to(const sv::ToArgs& a, hipStream_t s) {
  launch_stats_wave<E>(a.rows, const_cast<sv::RowStat*>(a.stats), int64_t{a.B} * (a.K + 1), s);
  hipLaunchKernelGGL((sv::to_verify_kernel<E, kStep, kStep>), dim3(static_cast<unsigned>(a.B)), dim3(sv::kThreads), 0,
                     s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

template <class E>
spec_status launch_sample(const sv::SampleArgs& a, hipStream_t s) {
  launch_stats_wave<E>(a.rows, const_cast<sv::RowStat*>(a.stats), int64_t{a.R}, s);
  hipLaunchKernelGGL((sv::sample_kernel<E, kStep, kStep>), dim3(static_cast<unsigned>(a.R)), dim3(sv::kThreads), 0,
                     s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

// Diagnostics per sub-chunk of kStep tiles, one wave per sub-chunk in both
// streaming passes.
template <class E>
spec_status launch_diag(const sv::DiagArgs& a, hipStream_t s) {
  const int C = a.rows.C;
  const int64_t units = int64_t{a.B} * a.K;
  const int64_t nsub = 2 * units * C;
  hipLaunchKernelGGL((sv::diag_stats_wave_kernel<E, kStep, kDiagStatVec>),
                     dim3(static_cast<unsigned>((nsub + sv::kWaves - 1) / sv::kWaves)), dim3(sv::kThreads), 0, s,
                     a.rows, const_cast<sv::DiagStat*>(a.stats), nsub);
  hipLaunchKernelGGL(sv::diag_norm_kernel, dim3(static_cast<unsigned>((2 * units + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a.stats, static_cast<int>(2 * units), C, a.norms, a.info);
  hipLaunchKernelGGL((sv::diag_pair_wave_kernel<E, kStep, kDiagPairVec>),
                     dim3(static_cast<unsigned>((units * C + sv::kWaves - 1) / sv::kWaves)), dim3(sv::kThreads), 0,
                     s, a, units * C);
  hipLaunchKernelGGL((sv::diag_finish_kernel<E>), dim3(static_cast<unsigned>((units + sv::kWaves - 1) / sv::kWaves)),
                     dim3(sv::kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SPEC_OK : SPEC_EHIP;
}

// Validation and argument block shared by the two verification entry points.
spec_status prepare_verify(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                           const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k, spec_dtype dtype,
                           int B, int K, int V, const int32_t* draft_ids, const float* temperature,
                           float temperature_scalar, uint64_t seed, uint64_t offset, int32_t* accept_len,
                           int32_t* emitted_ids, float* overlap, float* p_at_draft, float* q_at_draft,
                           float* logz_target, float* logz_draft, void* workspace, size_t workspace_bytes,
                           bool gumbel, sv::VerifyArgs* out, sv::GumbelBest** gbest) {
  // ---- validation: synchronous, before anything touches the GPU ------------
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (K > SPEC_MAX_K) return SPEC_EUNSUPPORTED;
  if (!verify_sizes_ok(B, K, V, dtype)) return SPEC_EINVAL;
  if (!target_logits || !draft_logits || !draft_ids || !accept_len || !emitted_ids) return SPEC_EINVAL;
  if (t_stride_b < 0 || t_stride_k < 0 || d_stride_b < 0 || d_stride_k < 0) return SPEC_EINVAL;
  if (!extent_ok(target_logits, B, t_stride_b, K + 1, t_stride_k, V, esize_of(dtype)) ||
      !extent_ok(draft_logits, B, d_stride_b, K, d_stride_k, V, esize_of(dtype)))
    return SPEC_EINVAL;
  if (!temperature && !(temperature_scalar > 0.f && std::isfinite(temperature_scalar))) return SPEC_EINVAL;
  const VerifyLayout L = verify_layout(B, K, V, dtype, gumbel);
  if (!workspace) return SPEC_EWORKSPACE;
  if (workspace_bytes < L.total) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  const size_t es = esize_of(dtype);
  sv::VerifyArgs a{};
  a.rows.tgt = target_logits; a.rows.tsb = t_stride_b; a.rows.tsk = t_stride_k; a.rows.tper = K + 1;
  a.rows.drf = draft_logits; a.rows.dsb = d_stride_b; a.rows.dsk = d_stride_k; a.rows.dper = K;
  a.rows.nb = B;
  a.rows.temp = temperature; a.rows.temp_scalar = temperature_scalar;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = gumbel ? g.C : sub_chunks(V, dtype);
  a.rows.vec_t = rows_vec_aligned(target_logits, t_stride_b, t_stride_k, es) ? 1 : 0;
  a.rows.vec_d = rows_vec_aligned(draft_logits, d_stride_b, d_stride_k, es) ? 1 : 0;
  a.B = B; a.K = K;
  a.ids = draft_ids;
  a.seed = seed; a.offset = offset;
  a.accept_len = accept_len; a.emitted = emitted_ids;
  a.overlap = overlap; a.p_at = p_at_draft; a.q_at = q_at_draft;
  a.logz_t = logz_target; a.logz_d = logz_draft;
  char* ws = static_cast<char*>(workspace);
  a.stats = reinterpret_cast<const sv::RowStat*>(ws + L.stats);
  a.norms = reinterpret_cast<sv::RowNorm*>(ws + L.norms);
  a.decision = reinterpret_cast<int32_t*>(ws + L.decision);
  a.pairs = reinterpret_cast<sv::PairStat*>(ws + L.pairs);
  a.want_z = gumbel ? 0 : 1;
  *gbest = gumbel ? reinterpret_cast<sv::GumbelBest*>(ws + L.gbest) : nullptr;
  *out = a;
  return SPEC_OK;
}

// ---- scratch memory for spec_verify_noalloc -------------------------------
// The workspace of spec_verify_noalloc: a file-scope device array, one copy
// on every GPU the library runs on, held until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol); it uses the device address that
// hipGetSymbolAddress returns, once per device, with that device current.
constexpr size_t kScratchBytes = size_t{32} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

void* g_scratch_ptr[kMaxDevices] = {};
std::atomic<int> g_scratch_ready[kMaxDevices] = {};
std::mutex g_scratch_mu;

// The current device's address of `scratch`, or nullptr on failure.
void* scratch_ptr() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  if (g_scratch_ready[dev].load(std::memory_order_acquire)) return g_scratch_ptr[dev];
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ready[dev].load(std::memory_order_relaxed)) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
    g_scratch_ready[dev].store(1, std::memory_order_release);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int spec_version(void) { return SPEC_VERSION; }

const char* spec_status_string(spec_status s) {
  switch (s) {
    case SPEC_OK: return "ok";
    case SPEC_EINVAL: return "invalid argument";
    case SPEC_EUNSUPPORTED: return "unsupported dtype or shape";
    case SPEC_EWORKSPACE: return "workspace missing or too small";
    case SPEC_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t spec_verify_workspace_size(int B, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!verify_sizes_ok(B, K, V, dtype)) return 0;
  return verify_layout(B, K, V, dtype).total;
}

size_t spec_tv_workspace_size(int N, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!tv_sizes_ok(N, K, V, dtype)) return 0;
  return tv_layout(N, K, V, dtype).total;
}


spec_status spec_verify(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                        const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                        spec_dtype dtype, int B, int K, int V, const int32_t* draft_ids,
                        const float* temperature, float temperature_scalar, uint64_t seed,
                        uint64_t offset, int32_t* accept_len, int32_t* emitted_ids, float* overlap,
                        float* p_at_draft, float* q_at_draft, float* logz_target, float* logz_draft,
                        void* workspace, size_t workspace_bytes, void* stream) {
  return spec_verify_ex(target_logits, t_stride_b, t_stride_k, draft_logits, d_stride_b, d_stride_k, dtype, B, K, V,
                        draft_ids, temperature, temperature_scalar, seed, offset, accept_len, emitted_ids, overlap,
                        p_at_draft, q_at_draft, logz_target, logz_draft, workspace, workspace_bytes, stream, nullptr);
}

spec_status spec_verify_ex(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                           const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                           spec_dtype dtype, int B, int K, int V, const int32_t* draft_ids,
                           const float* temperature, float temperature_scalar, uint64_t seed,
                           uint64_t offset, int32_t* accept_len, int32_t* emitted_ids, float* overlap,
                           float* p_at_draft, float* q_at_draft, float* logz_target, float* logz_draft,
                           void* workspace, size_t workspace_bytes, void* stream, const spec_launch* launch) {
  if (launch && (launch->path < SPEC_PATH_AUTO || launch->path > SPEC_PATH_SINGLE_READ || launch->groups < 0 ||
                 launch->residual_shape < 0 || launch->residual_shape > 2))
    return SPEC_EINVAL;
  sv::VerifyArgs a;
  sv::GumbelBest* gb;
  const spec_status st = prepare_verify(target_logits, t_stride_b, t_stride_k, draft_logits, d_stride_b, d_stride_k,
                                        dtype, B, K, V, draft_ids, temperature, temperature_scalar, seed, offset,
                                        accept_len, emitted_ids, overlap, p_at_draft, q_at_draft, logz_target,
                                        logz_draft, workspace, workspace_bytes, false, &a, &gb);
  if (st != SPEC_OK) return st;
  const int64_t rows = int64_t{B} * (2 * K + 1);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_verify<BF16>(a, rows, s, launch) : launch_verify<F32>(a, rows, s, launch);
}

size_t spec_verify_noalloc_max_workspace(void) { return kScratchBytes; }

spec_status spec_verify_noalloc(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                                const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                                spec_dtype dtype, int B, int K, int V, const int32_t* draft_ids,
                                const float* temperature, float temperature_scalar, uint64_t seed,
                                uint64_t offset, int32_t* accept_len, int32_t* emitted_ids, float* overlap,
                                float* p_at_draft, float* q_at_draft, float* logz_target, float* logz_draft,
                                void* stream) {
  const size_t need = spec_verify_workspace_size(B, K, V, dtype);
  if (need > kScratchBytes) return SPEC_EWORKSPACE;  // beyond the scratch array (also: need 0 is checked below)
  // a first pass over the arguments (with a stand-in workspace address that is
  // never used) returns argument errors before the scratch address is looked
  // up, so a bad call does not touch the GPU
  sv::VerifyArgs a;
  sv::GumbelBest* gb;
  spec_status st = prepare_verify(target_logits, t_stride_b, t_stride_k, draft_logits, d_stride_b, d_stride_k,
                                  dtype, B, K, V, draft_ids, temperature, temperature_scalar, seed, offset,
                                  accept_len, emitted_ids, overlap, p_at_draft, q_at_draft, logz_target,
                                  logz_draft, reinterpret_cast<void*>(uintptr_t{256}), kScratchBytes, false, &a,
                                  &gb);
  if (st != SPEC_OK) return st;
  void* ws = scratch_ptr();
  if (!ws) return SPEC_EHIP;
  st = prepare_verify(target_logits, t_stride_b, t_stride_k, draft_logits, d_stride_b, d_stride_k, dtype, B, K, V,
                      draft_ids, temperature, temperature_scalar, seed, offset, accept_len, emitted_ids, overlap,
                      p_at_draft, q_at_draft, logz_target, logz_draft, ws, kScratchBytes, false, &a, &gb);
  if (st != SPEC_OK) return st;
  const int64_t rows = int64_t{B} * (2 * K + 1);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_verify<BF16>(a, rows, s) : launch_verify<F32>(a, rows, s);
}

size_t spec_verify_gumbel_workspace_size(int B, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!verify_sizes_ok(B, K, V, dtype)) return 0;
  return verify_layout(B, K, V, dtype, true).total;
}

spec_status spec_verify_gumbel(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                               const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k,
                               spec_dtype dtype, int B, int K, int V, const int32_t* draft_ids,
                               const float* temperature, float temperature_scalar, uint64_t seed,
                               uint64_t offset, int32_t* accept_len, int32_t* emitted_ids, float* overlap,
                               float* p_at_draft, float* q_at_draft, float* logz_target, float* logz_draft,
                               void* workspace, size_t workspace_bytes, void* stream) {
  sv::VerifyArgs a;
  sv::GumbelBest* gb;
  const spec_status st = prepare_verify(target_logits, t_stride_b, t_stride_k, draft_logits, d_stride_b, d_stride_k,
                                        dtype, B, K, V, draft_ids, temperature, temperature_scalar, seed, offset,
                                        accept_len, emitted_ids, overlap, p_at_draft, q_at_draft, logz_target,
                                        logz_draft, workspace, workspace_bytes, true, &a, &gb);
  if (st != SPEC_OK) return st;
  const int64_t rows = int64_t{B} * (2 * K + 1);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_verify_gumbel<BF16, kNtBf16>(a, gb, rows, s)
                            : launch_verify_gumbel<F32, kNtF32>(a, gb, rows, s);
}

size_t spec_sample_gumbel_workspace_size(int R, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!rows_ok(R, V, dtype)) return 0;
  return align_up(static_cast<size_t>(R) * geometry(V, dtype).C * sizeof(sv::GumbelBest), 256);
}

spec_status spec_sample_gumbel(const void* logits, int64_t stride_r, spec_dtype dtype, int R, int V,
                               const float* temperature, float temperature_scalar, uint64_t seed, uint64_t offset,
                               int32_t* tokens, void* workspace, size_t workspace_bytes, void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (!rows_ok(R, V, dtype)) return SPEC_EINVAL;
  if (!logits || !tokens || stride_r < 0) return SPEC_EINVAL;
  if (!extent_ok(logits, R, stride_r, 1, 0, V, esize_of(dtype))) return SPEC_EINVAL;
  if (!temperature && !(temperature_scalar >= 0.f && std::isfinite(temperature_scalar))) return SPEC_EINVAL;
  if (!workspace || workspace_bytes < spec_sample_gumbel_workspace_size(R, V, dtype)) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  sv::GumbelSampleArgs a{};
  a.rows.tgt = logits; a.rows.tsb = stride_r; a.rows.tsk = 0; a.rows.tper = 1;
  a.rows.drf = nullptr; a.rows.dsb = 0; a.rows.dsk = 0; a.rows.dper = 1;
  a.rows.nb = R;
  a.rows.temp = temperature; a.rows.temp_scalar = temperature_scalar;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = g.C;
  a.rows.vec_t = rows_vec_aligned(logits, stride_r, 0, esize_of(dtype)) ? 1 : 0;
  a.rows.vec_d = 0;
  a.R = R;
  a.seed = seed; a.offset = offset;
  a.token = tokens;
  a.best = reinterpret_cast<sv::GumbelBest*>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_sample_gumbel<BF16, kNtBf16>(a, s) : launch_sample_gumbel<F32, kNtF32>(a, s);
}

spec_status spec_tv_loss_fwd_bwd(const void* target_logits, int64_t t_stride_n, int64_t t_stride_k,
                                 const void* draft_logits, int64_t d_stride_n, int64_t d_stride_k,
                                 spec_dtype dtype, int N, int K, int V, float temperature, spec_tv_mode mode,
                                 float scale, float* loss, float* overlap, float* grad_draft, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (K > SPEC_MAX_K) return SPEC_EUNSUPPORTED;
  if (!tv_sizes_ok(N, K, V, dtype)) return SPEC_EINVAL;
  if (!target_logits || !draft_logits || !loss) return SPEC_EINVAL;
  if (t_stride_n < 0 || t_stride_k < 0 || d_stride_n < 0 || d_stride_k < 0) return SPEC_EINVAL;
  if (!extent_ok(target_logits, N, t_stride_n, K, t_stride_k, V, esize_of(dtype)) ||
      !extent_ok(draft_logits, N, d_stride_n, K, d_stride_k, V, esize_of(dtype)))
    return SPEC_EINVAL;
  if (!(temperature > 0.f && std::isfinite(temperature))) return SPEC_EINVAL;
  if (mode != SPEC_TV_E2E && mode != SPEC_TV_PROD && mode != SPEC_TV_PER_STEP) return SPEC_EINVAL;
  if (!std::isfinite(scale)) return SPEC_EINVAL;
  const TvLayout L = tv_layout(N, K, V, dtype);
  if (!workspace) return SPEC_EWORKSPACE;
  if (workspace_bytes < L.total) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  const size_t es = esize_of(dtype);
  sv::TvArgs a{};
  a.rows.tgt = target_logits; a.rows.tsb = t_stride_n; a.rows.tsk = t_stride_k; a.rows.tper = K;
  a.rows.drf = draft_logits; a.rows.dsb = d_stride_n; a.rows.dsk = d_stride_k; a.rows.dper = K;
  a.rows.nb = N;
  a.rows.temp = nullptr; a.rows.temp_scalar = temperature;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = g.C;
  a.rows.vec_t = rows_vec_aligned(target_logits, t_stride_n, t_stride_k, es) ? 1 : 0;
  a.rows.vec_d = rows_vec_aligned(draft_logits, d_stride_n, d_stride_k, es) ? 1 : 0;
  a.N = N; a.K = K;
  a.mode = static_cast<int>(mode);
  a.scale = static_cast<double>(scale);
  a.inv_t = 1.0f / temperature;
  a.loss = loss; a.overlap = overlap; a.grad = grad_draft;
  char* ws = static_cast<char*>(workspace);
  a.stats = reinterpret_cast<const sv::RowStat*>(ws + L.stats);
  a.norms = reinterpret_cast<const sv::RowNorm*>(ws + L.norms);
  a.pairs = reinterpret_cast<sv::TvPair*>(ws + L.pairs);
  a.coef = reinterpret_cast<float2*>(ws + L.coef);
  a.loss_pos = reinterpret_cast<double*>(ws + L.loss);
  a.vec_g = (grad_draft && aligned16(grad_draft) && (V % 4 == 0)) ? 1 : 0;
  a.bits = grad_draft ? reinterpret_cast<uint8_t*>(ws + L.bits) : nullptr;
  a.bits_stride = static_cast<int64_t>(L.bits_stride);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_tv<BF16, kNtBf16>(a, s) : launch_tv<F32, kNtF32>(a, s);
}

size_t spec_verify_target_only_workspace_size(int B, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (B < 1 || K < 1 || K > SPEC_MAX_K || !rows_sub_ok(int64_t{B} * (K + 1), V, dtype)) return 0;
  return to_layout(B, K, V, dtype).total;
}

spec_status spec_verify_target_only(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                                    spec_dtype dtype, int B, int K, int V, const int32_t* draft_ids,
                                    const float* temperature, float temperature_scalar, uint64_t seed,
                                    uint64_t offset, int32_t* accept_len, int32_t* emitted_ids, float* p_at_draft,
                                    float* logz_target, void* workspace, size_t workspace_bytes, void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (K > SPEC_MAX_K) return SPEC_EUNSUPPORTED;
  if (B < 1 || K < 1 || !rows_sub_ok(int64_t{B} * (K + 1), V, dtype)) return SPEC_EINVAL;
  if (!target_logits || !draft_ids || !accept_len || !emitted_ids) return SPEC_EINVAL;
  if (t_stride_b < 0 || t_stride_k < 0) return SPEC_EINVAL;
  if (!extent_ok(target_logits, B, t_stride_b, K + 1, t_stride_k, V, esize_of(dtype))) return SPEC_EINVAL;
  if (!temperature && !(temperature_scalar > 0.f && std::isfinite(temperature_scalar))) return SPEC_EINVAL;
  const ToLayout L = to_layout(B, K, V, dtype);
  if (!workspace || workspace_bytes < L.total) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  sv::ToArgs a{};
  a.rows.tgt = target_logits; a.rows.tsb = t_stride_b; a.rows.tsk = t_stride_k; a.rows.tper = K + 1;
  a.rows.drf = nullptr; a.rows.dsb = 0; a.rows.dsk = 0; a.rows.dper = 1;
  a.rows.nb = B;
  a.rows.temp = temperature; a.rows.temp_scalar = temperature_scalar;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = sub_chunks(V, dtype);
  a.rows.vec_t = rows_vec_aligned(target_logits, t_stride_b, t_stride_k, esize_of(dtype)) ? 1 : 0;
  a.rows.vec_d = 0;
  a.B = B; a.K = K;
  a.ids = draft_ids;
  a.seed = seed; a.offset = offset;
  a.accept_len = accept_len; a.emitted = emitted_ids; a.p_at = p_at_draft; a.logz_t = logz_target;
  a.stats = reinterpret_cast<const sv::RowStat*>(static_cast<char*>(workspace) + L.stats);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_to<BF16>(a, s) : launch_to<F32>(a, s);
}

size_t spec_sample_workspace_size(int R, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!rows_sub_ok(R, V, dtype)) return 0;
  return sample_ws(R, V, dtype);
}

spec_status spec_sample(const void* logits, int64_t stride_r, spec_dtype dtype, int R, int V,
                        const float* temperature, float temperature_scalar, uint64_t seed, uint64_t offset,
                        int32_t* tokens, float* logz, void* workspace, size_t workspace_bytes, void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (!rows_sub_ok(R, V, dtype)) return SPEC_EINVAL;
  if (!logits || !tokens || stride_r < 0) return SPEC_EINVAL;
  if (!extent_ok(logits, R, stride_r, 1, 0, V, esize_of(dtype))) return SPEC_EINVAL;
  if (!temperature && !(temperature_scalar >= 0.f && std::isfinite(temperature_scalar))) return SPEC_EINVAL;
  if (!workspace || workspace_bytes < sample_ws(R, V, dtype)) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  sv::SampleArgs a{};
  a.rows.tgt = logits; a.rows.tsb = stride_r; a.rows.tsk = 0; a.rows.tper = 1;
  a.rows.drf = nullptr; a.rows.dsb = 0; a.rows.dsk = 0; a.rows.dper = 1;
  a.rows.nb = R;
  a.rows.temp = temperature; a.rows.temp_scalar = temperature_scalar;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = sub_chunks(V, dtype);
  a.rows.vec_t = rows_vec_aligned(logits, stride_r, 0, esize_of(dtype)) ? 1 : 0;
  a.rows.vec_d = 0;
  a.R = R;
  a.seed = seed; a.offset = offset;
  a.token = tokens; a.logz = logz;
  a.stats = reinterpret_cast<const sv::RowStat*>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_sample<BF16>(a, s) : launch_sample<F32>(a, s);
}

size_t spec_diagnostics_workspace_size(int B, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (B < 1 || K < 1 || K > SPEC_MAX_K || !rows_sub_ok(int64_t{B} * 2 * K, V, dtype)) return 0;
  return diag_layout(B, K, V, dtype).total;
}

spec_status spec_diagnostics(const void* target_logits, int64_t t_stride_b, int64_t t_stride_k,
                             const void* draft_logits, int64_t d_stride_b, int64_t d_stride_k, spec_dtype dtype,
                             int B, int K, int V, const float* temperature, float temperature_scalar, float* diag,
                             int32_t* greedy_draft, int32_t* rs_preferred, void* workspace, size_t workspace_bytes,
                             void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (K > SPEC_MAX_K) return SPEC_EUNSUPPORTED;
  if (B < 1 || K < 1 || !rows_sub_ok(int64_t{B} * 2 * K, V, dtype)) return SPEC_EINVAL;
  if (!target_logits || !draft_logits || !diag) return SPEC_EINVAL;
  if (t_stride_b < 0 || t_stride_k < 0 || d_stride_b < 0 || d_stride_k < 0) return SPEC_EINVAL;
  if (!extent_ok(target_logits, B, t_stride_b, K, t_stride_k, V, esize_of(dtype)) ||
      !extent_ok(draft_logits, B, d_stride_b, K, d_stride_k, V, esize_of(dtype)))
    return SPEC_EINVAL;
  if (!temperature && !(temperature_scalar > 0.f && std::isfinite(temperature_scalar))) return SPEC_EINVAL;
  const DiagLayout L = diag_layout(B, K, V, dtype);
  if (!workspace || workspace_bytes < L.total) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  const size_t es = esize_of(dtype);
  sv::DiagArgs a{};
  a.rows.tgt = target_logits; a.rows.tsb = t_stride_b; a.rows.tsk = t_stride_k; a.rows.tper = K;
  a.rows.drf = draft_logits; a.rows.dsb = d_stride_b; a.rows.dsk = d_stride_k; a.rows.dper = K;
  a.rows.nb = B;
  a.rows.temp = temperature; a.rows.temp_scalar = temperature_scalar;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = sub_chunks(V, dtype);
  a.rows.vec_t = rows_vec_aligned(target_logits, t_stride_b, t_stride_k, es) ? 1 : 0;
  a.rows.vec_d = rows_vec_aligned(draft_logits, d_stride_b, d_stride_k, es) ? 1 : 0;
  a.B = B; a.K = K;
  a.out = diag; a.greedy = greedy_draft; a.prefer = rs_preferred;
  char* ws = static_cast<char*>(workspace);
  a.stats = reinterpret_cast<const sv::DiagStat*>(ws + L.stats);
  a.norms = reinterpret_cast<sv::RowNorm*>(ws + L.norms);
  a.info = reinterpret_cast<sv::DiagRow*>(ws + L.info);
  a.pairs = reinterpret_cast<sv::DiagPair*>(ws + L.pairs);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_diag<BF16>(a, s) : launch_diag<F32>(a, s);
}

size_t spec_kl_workspace_size(int N, int K, int V, spec_dtype dtype) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return 0;
  if (!tv_sizes_ok(N, K, V, dtype)) return 0;
  return kl_layout(N, K, V, dtype).total;
}

spec_status spec_kl_loss_fwd_bwd(const void* target_logits, int64_t t_stride_n, int64_t t_stride_k,
                                 const void* draft_logits, int64_t d_stride_n, int64_t d_stride_k,
                                 spec_dtype dtype, int N, int K, int V, float temperature, spec_kl_kind kind,
                                 float scale, float* loss, float* per_step, float* grad_draft, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  if (dtype != SPEC_F32 && dtype != SPEC_BF16) return SPEC_EUNSUPPORTED;
  if (K > SPEC_MAX_K) return SPEC_EUNSUPPORTED;
  if (!tv_sizes_ok(N, K, V, dtype)) return SPEC_EINVAL;
  if (!target_logits || !draft_logits || !loss) return SPEC_EINVAL;
  if (t_stride_n < 0 || t_stride_k < 0 || d_stride_n < 0 || d_stride_k < 0) return SPEC_EINVAL;
  if (!extent_ok(target_logits, N, t_stride_n, K, t_stride_k, V, esize_of(dtype)) ||
      !extent_ok(draft_logits, N, d_stride_n, K, d_stride_k, V, esize_of(dtype)))
    return SPEC_EINVAL;
  if (!(temperature > 0.f && std::isfinite(temperature))) return SPEC_EINVAL;
  if (kind != SPEC_KL_FORWARD && kind != SPEC_KL_CE && kind != SPEC_KL_REVERSE) return SPEC_EINVAL;
  if (!std::isfinite(scale)) return SPEC_EINVAL;
  const KlLayout L = kl_layout(N, K, V, dtype);
  if (!workspace || workspace_bytes < L.total) return SPEC_EWORKSPACE;
  if (!aligned16(workspace)) return SPEC_EINVAL;

  const Geometry g = geometry(V, dtype);
  const size_t es = esize_of(dtype);
  sv::KlArgs a{};
  a.rows.tgt = target_logits; a.rows.tsb = t_stride_n; a.rows.tsk = t_stride_k; a.rows.tper = K;
  a.rows.drf = draft_logits; a.rows.dsb = d_stride_n; a.rows.dsk = d_stride_k; a.rows.dper = K;
  a.rows.nb = N;
  a.rows.temp = nullptr; a.rows.temp_scalar = temperature;
  a.rows.V = V; a.rows.ntiles = g.ntiles; a.rows.C = g.C;
  a.rows.vec_t = rows_vec_aligned(target_logits, t_stride_n, t_stride_k, es) ? 1 : 0;
  a.rows.vec_d = rows_vec_aligned(draft_logits, d_stride_n, d_stride_k, es) ? 1 : 0;
  a.N = N; a.K = K;
  a.kind = static_cast<int>(kind);
  a.scale = static_cast<double>(scale);
  a.inv_t = 1.0f / temperature;
  a.loss = loss; a.per_step = per_step; a.grad = grad_draft;
  char* ws = static_cast<char*>(workspace);
  a.stats = reinterpret_cast<sv::KlStat*>(ws + L.stats);
  a.SC = sub_chunks(V, dtype);
  a.norms = reinterpret_cast<sv::KlNorm*>(ws + L.norms);
  a.parts = reinterpret_cast<sv::KlPart*>(ws + L.parts);
  a.coef = reinterpret_cast<float4*>(ws + L.coef);
  a.loss_pos = reinterpret_cast<double*>(ws + L.loss);
  // lam_t - lam_d = log2(max q / max p); beyond the limit the separately
  // summed normalisers (error a few 1e-7) move the gradient by at most
  // 64 (bfloat16) or 3.4 (float32) times that error against the row's
  // largest |q - p|, far inside the tolerances (2e-3, 1e-5)
  a.pair_limit = dtype == SPEC_BF16 ? 1.0 / 64 : 0.5;
  a.vec_g = (grad_draft && aligned16(grad_draft) && (V % 4 == 0)) ? 1 : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == SPEC_BF16 ? launch_kl_kind<BF16, kNtBf16>(a, s) : launch_kl_kind<F32, kNtF32>(a, s);
}

}  // extern "C"

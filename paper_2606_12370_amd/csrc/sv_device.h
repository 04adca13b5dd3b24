// sv_device.h — device building blocks for the gfx950 verification and
// TV-loss kernels: element types, 16-byte row loads, Philox4x64-10, wave64
// and workgroup reductions and scans, and the per-chunk row statistics that
// every kernel combines into a row's log2 normaliser.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sv {

constexpr int kThreads = 256;          // one workgroup = 4 wave64
constexpr int kWaves = kThreads / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLog2eD = 1.4426950408889634074;
constexpr double kLn2D = 0.69314718055994530942;
#define SPEC_MAX_K_DEV 8

// 16-byte vector types the compiler treats as native vectors (needed by the
// non-temporal load / store builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Element types: logits arrive as bfloat16 bit patterns or float32.  Each
// thread owns one vector per tile, i.e. EPV consecutive elements, loaded with
// one instruction.  BF16 and F32 use 16-byte vectors; BF16H reads bfloat16
// as 8-byte vectors of 4, so that a pass writing one float32 per element
// stores one contiguous 16-byte vector per lane.
struct BF16 {
  using raw = uint16_t;
  using vec = u32x4;
  static constexpr int EPV = 8;
  static constexpr bool kFoldRef = true;  // the overlap may fold M + L into one constant
  static __device__ __forceinline__ void widen(const vec v, float (&x)[8]) {
    x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xffff0000u);
    x[4] = __uint_as_float(v.z << 16); x[5] = __uint_as_float(v.z & 0xffff0000u);
    x[6] = __uint_as_float(v.w << 16); x[7] = __uint_as_float(v.w & 0xffff0000u);
  }
  static __device__ __forceinline__ float one(const raw* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
};

struct BF16H {
  using raw = uint16_t;
  using vec = u32x2;
  static constexpr int EPV = 4;
  static constexpr bool kFoldRef = true;
  static __device__ __forceinline__ void widen(const vec v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xffff0000u);
  }
  static __device__ __forceinline__ float one(const raw* p) { return BF16::one(p); }
};

struct F32 {
  using raw = float;
  using vec = u32x4;
  static constexpr int EPV = 4;
  static constexpr bool kFoldRef = false;
  static __device__ __forceinline__ void widen(const vec v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
    x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  static __device__ __forceinline__ float one(const raw* p) { return *p; }
};

// Load S vectors of a span read by W lanes together: x[j][k] receives element
// e0 + j * W * EPV + idx * EPV + k of the row (idx: this lane's index among
// the W).  Elements at or beyond V are -inf (probability 0).  With `aligned`
// (row base 16-byte aligned) every full vector is one vector load, all issued
// back to back; a vector past V is read from the row start and discarded (no
// branch around the load); the one vector that straddles V (V not a multiple
// of EPV) is completed element by element.  Unaligned rows are read element
// by element.
template <class E, int S, int W>
__device__ __forceinline__ void load_span(const typename E::raw* __restrict__ row, int e0, int idx, int V,
                                          bool aligned, float (&x)[S][E::EPV]) {
  constexpr int EPV = E::EPV;
  if (aligned) {
    typename E::vec w[S];
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const int v0 = e0 + j * W * EPV + idx * EPV;
      const int off = (v0 + EPV <= V) ? v0 : 0;
      w[j] = __builtin_nontemporal_load(reinterpret_cast<const typename E::vec*>(row + off));
    }
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const int v0 = e0 + j * W * EPV + idx * EPV;
      E::widen(w[j], x[j]);
      if (v0 + EPV > V) {
#pragma unroll
        for (int k = 0; k < EPV; ++k) x[j][k] = (v0 + k < V) ? E::one(row + v0 + k) : -INFINITY;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const int v0 = e0 + j * W * EPV + idx * EPV;
#pragma unroll
      for (int k = 0; k < EPV; ++k) x[j][k] = (v0 + k < V) ? E::one(row + v0 + k) : -INFINITY;
    }
  }
}

// Load S tiles (tile0 .. tile0+S-1) of a row, a tile being one vector of each
// of the workgroup's 256 threads: x[j][k] receives element
// (tile0 + j) * 256 * EPV + t * EPV + k of the row, t = threadIdx.x.
template <class E, int S>
__device__ __forceinline__ void load_tiles(const typename E::raw* __restrict__ row, int tile0, int V, bool aligned,
                                           float (&x)[S][E::EPV]) {
  load_span<E, S, 256>(row, tile0 * 256 * E::EPV, static_cast<int>(threadIdx.x), V, aligned, x);
}

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Counter (c0..c3), key
// (k0, k1); each round multiplies c0 and c2 by the two published multipliers,
// mixes the high halves with c1 / c3 and the key, and the key is bumped by the
// two Weyl constants between rounds.
struct Philox4x64 {
  uint64_t w[4];
};
// Full 128-bit product a * m as (hi, lo), schoolbook over 32-bit halves: four
// 32 x 32 -> 64-bit partial products; a partial plus the 32-bit carries added
// to it stays below 2^64 ((2^32 - 1)^2 + 2 (2^32 - 1) = 2^64 - 1), so both
// halves come from four multiply-adds and one add.
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t m, uint64_t* lo, uint64_t* hi) {
  const uint64_t a0 = static_cast<uint32_t>(a), a1 = a >> 32;
  const uint64_t m0 = static_cast<uint32_t>(m), m1 = m >> 32;
  const uint64_t p00 = a0 * m0;
  const uint64_t p01 = a0 * m1 + (p00 >> 32);
  const uint64_t p10 = a1 * m0 + static_cast<uint32_t>(p01);
  *hi = a1 * m1 + (p01 >> 32) + (p10 >> 32);
  *lo = (p10 << 32) | static_cast<uint32_t>(p00);
}

__device__ inline Philox4x64 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                           uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += W0; k1 += W1; }
    uint64_t lo0, hi0, lo1, hi1;
    mulhilo64(c0, M0, &lo0, &hi0);
    mulhilo64(c2, M1, &lo1, &hi1);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
  Philox4x64 out;
  out.w[0] = c0; out.w[1] = c1; out.w[2] = c2; out.w[3] = c3;
  return out;
}

// Top 24 bits as a uniform on the 2^-24 grid in [0, 1) (exact in float32).
__device__ __forceinline__ double u24(uint64_t w) {
  return static_cast<double>(w >> 40) * (1.0 / 16777216.0);
}

// ---------------------------------------------------------------------------
// wave64 and workgroup reductions / scans.  All reductions run in a fixed
// order so results are bitwise reproducible.
//
// The max and sum reductions use DPP lane permutations inside each row of 16
// lanes (a butterfly: swap neighbours, swap pairs, mirror the half row,
// mirror the row; a commutative step gives every lane of the row the same
// bits) and then combine the four rows' results, read from lanes 0, 16, 32
// and 48, in a fixed order.  No LDS traffic is involved.
namespace dpp {
constexpr int kXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror: lane i <- 7 - i within 8
constexpr int kMirror = 0x140;      // row_mirror: lane i <- 15 - i within 16
template <int CTRL>
__device__ __forceinline__ float mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
template <int CTRL>
__device__ __forceinline__ double mov(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(b), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(b >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
__device__ __forceinline__ float lane(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double lane(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(b), l);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), l);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
}  // namespace dpp

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp::mov<dpp::kXor1>(v));
  v = fmaxf(v, dpp::mov<dpp::kXor2>(v));
  v = fmaxf(v, dpp::mov<dpp::kHalfMirror>(v));
  v = fmaxf(v, dpp::mov<dpp::kMirror>(v));
  return fmaxf(fmaxf(dpp::lane(v, 0), dpp::lane(v, 16)), fmaxf(dpp::lane(v, 32), dpp::lane(v, 48)));
}
__device__ __forceinline__ double wave_sum(double v) {
  v += dpp::mov<dpp::kXor1>(v);
  v += dpp::mov<dpp::kXor2>(v);
  v += dpp::mov<dpp::kHalfMirror>(v);
  v += dpp::mov<dpp::kMirror>(v);
  return (dpp::lane(v, 0) + dpp::lane(v, 16)) + (dpp::lane(v, 32) + dpp::lane(v, 48));
}
__device__ __forceinline__ int wave_min_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}
// inclusive scan over the 64 lanes of a wave
__device__ __forceinline__ double wave_incl_scan(double v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

// Scratch for workgroup-wide reductions (lives in LDS).
template <int N>
struct RedLds {
  double d[kWaves][N];
  float f[kWaves][N];
  int i[kWaves];
};

// Workgroup max of N floats per thread; every thread receives the results.
template <int N>
__device__ __forceinline__ void wg_max(float (&v)[N], RedLds<N>& s) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] = wave_max(v[n]);
  if (lane == 0) {
#pragma unroll
    for (int n = 0; n < N; ++n) s.f[wave][n] = v[n];
  }
  __syncthreads();
#pragma unroll
  for (int n = 0; n < N; ++n) {
    float m = s.f[0][n];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = fmaxf(m, s.f[w][n]);
    v[n] = m;
  }
  __syncthreads();
}

// Workgroup sum of N doubles per thread; every thread receives the results.
template <int N>
__device__ __forceinline__ void wg_sum(double (&v)[N], RedLds<N>& s) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] = wave_sum(v[n]);
  if (lane == 0) {
#pragma unroll
    for (int n = 0; n < N; ++n) s.d[wave][n] = v[n];
  }
  __syncthreads();
#pragma unroll
  for (int n = 0; n < N; ++n) {
    double a = s.d[0][n];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) a += s.d[w][n];
    v[n] = a;
  }
  __syncthreads();
}


// Workgroup minimum of an int (every thread receives it).
__device__ __forceinline__ int wg_min_int(int v, RedLds<1>& s) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  v = wave_min_int(v);
  if (lane == 0) s.i[wave] = v;
  __syncthreads();
  int m = s.i[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) m = min(m, s.i[w]);
  __syncthreads();
  return m;
}

// ---------------------------------------------------------------------------
// Row statistics.  For a row z (logits) and s = log2(e) / T, the row's
// softmax is p_v = 2^(z_v s - M) / D with M a reference in log2 units and
// D = sum_v 2^(z_v s - M).  A chunk of the row reduces to (m_c, D_c): its
// largest per-thread reference and its sum relative to it.  References are
// rounded once (rs = round(max z * s)) and every exponent is formed as
// fma(z, s, -rs), so the exact product z*s enters each element and no
// per-thread rounding shift biases the normalised values.
struct RowStat {
  float m;     // largest thread reference of the chunk, log2 units (-inf: empty)
  float pad;
  double D;    // sum of 2^(z s - m) over the chunk
};

__host__ __device__ __forceinline__ float scale_of(float T) {
  return static_cast<float>(kLog2eD / static_cast<double>(T));
}

// Combine a row's C chunk statistics into (M, D).  Called by all 64 lanes of
// one wave; every lane receives the result.  The order of the float64 sum is
// fixed, so every kernel that combines the same row gets the same bits.
__device__ __forceinline__ void combine_row(const RowStat* __restrict__ st, int C, float* M, double* D) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY;
  for (int cc = lane; cc < C; cc += 64) m = fmaxf(m, st[cc].m);
  m = wave_max(m);
  double d = 0.0;
  for (int cc = lane; cc < C; cc += 64) {
    const float mc = st[cc].m;
    const double dc = st[cc].D;
    if (dc != dc) d += dc;
    else if (mc != -INFINITY) d += dc * static_cast<double>(__builtin_amdgcn_exp2f(mc - m));
  }
  *M = m;
  *D = wave_sum(d);
}

// combine_row for two rows at once (one wave), both rows' loads issued before
// either reduction; the sums run in combine_row's order, so each row gets the
// same bits as combine_row would give it.
__device__ __forceinline__ void combine_two_rows(const RowStat* __restrict__ s1, const RowStat* __restrict__ s2,
                                                 int C, float* M1, double* D1, float* M2, double* D2) {
  const int lane = threadIdx.x & 63;
  if (C > 64) {
    combine_row(s1, C, M1, D1);
    combine_row(s2, C, M2, D2);
    return;
  }
  RowStat a, b;
  a.m = -INFINITY; a.D = 0.0; b.m = -INFINITY; b.D = 0.0;
  if (lane < C) {
    a = s1[lane];
    b = s2[lane];
  }
  const float m1 = wave_max(a.m), m2 = wave_max(b.m);
  double d1 = 0.0, d2 = 0.0;
  if (lane < C) {
    if (a.D != a.D) d1 += a.D;
    else if (a.m != -INFINITY) d1 += a.D * static_cast<double>(__builtin_amdgcn_exp2f(a.m - m1));
    if (b.D != b.D) d2 += b.D;
    else if (b.m != -INFINITY) d2 += b.D * static_cast<double>(__builtin_amdgcn_exp2f(b.m - m2));
  }
  *M1 = m1;
  *D1 = wave_sum(d1);
  *M2 = m2;
  *D2 = wave_sum(d2);
}

// A row's combined normaliser: p_v = 2^(z_v s - M) / D.
struct RowNorm {
  float M;      // log2 units; +inf / NaN / -inf mark a bad row
  float invD;   // 1 / D rounded once
  float L;      // log2(D) rounded once
  float Llo;    // log2(D) - L, so that L + Llo carries log2(D) to about 2^-48
  double D;
};

__device__ __forceinline__ RowNorm make_norm(float M, double D) {
  RowNorm n;
  n.M = M;
  n.invD = static_cast<float>(1.0 / D);
  const double l2 = log2(D);
  n.L = static_cast<float>(l2);
  n.Llo = (l2 - l2 == 0.0) ? static_cast<float>(l2 - static_cast<double>(n.L)) : 0.f;  // 0 for D = 0 or inf
  n.D = D;
  return n;
}
__device__ __forceinline__ bool norm_ok(const RowNorm& n) { return n.D > 0.0 && n.D < INFINITY && n.M < INFINITY; }

// One wave per row: combine every row's chunk statistics (4 rows per
// 256-thread workgroup).
__global__ __launch_bounds__(kThreads) void row_norm_kernel(const RowStat* __restrict__ stats, int rows, int C,
                                                            RowNorm* __restrict__ out) {
  const int r = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (r >= rows) return;
  float M;
  double D;
  combine_row(stats + static_cast<int64_t>(r) * C, C, &M, &D);
  if ((threadIdx.x & 63) == 0) out[r] = make_norm(M, D);
}

// Probability of one element given its row's (M, 1/D): 2^(z s - M) / D.
__device__ __forceinline__ float prob(float z, float s, float M, float invD) {
  return __builtin_amdgcn_exp2f(fmaf(z, s, -M)) * invD;
}

// min(p, q) from one exponential: 2^(min(z_t s - M_t - L_t, z_d s - M_d - L_d)).
// One more rounding than prob() (L enters as a float), about 1e-6 relative.
__device__ __forceinline__ float min_prob(float zt, float zd, float s, const RowNorm& t, const RowNorm& d) {
  return __builtin_amdgcn_exp2f(fminf(fmaf(zt, s, -t.M) - t.L, fmaf(zd, s, -d.M) - d.L));
}

// min(p, q) with each row's reference and log2 normaliser folded into one
// float32 constant r = M + L: one rounding of r (about 6e-8 |r|, a few 1e-6
// relative for logits of size 100) against the two subtractions it saves;
// used for bfloat16 logits, whose tolerance is 2e-3.
__device__ __forceinline__ float min_prob_folded(float zt, float zd, float s, float rt, float rd) {
  return __builtin_amdgcn_exp2f(fminf(fmaf(zt, s, -rt), fmaf(zd, s, -rd)));
}

// The overlap term of element type E: folded references for bfloat16 logits.
template <class E>
__device__ __forceinline__ float overlap_term(float zt, float zd, float s, const RowNorm& t, const RowNorm& d,
                                              float rt, float rd) {
  if constexpr (E::kFoldRef) return min_prob_folded(zt, zd, s, rt, rd);
  else return min_prob(zt, zd, s, t, d);
}

// 1 - 2^-x for x >= 0: the series of -expm1(-y), y = x ln2, below x = 1/2
// (degree 9, truncation below 3e-10 of the value), the exponential above.
// 1 - 2^-x for 0 <= x < 1/2 from the series of 1 - e^-y, y = x ln 2 < 0.35,
// with the terms up to y^(D+1): truncation below y^(D+1) / (D+2)! of the
// value (D = 6: 6e-8, D = 3: 7e-6).
template <int D>
__device__ __forceinline__ float one_minus_exp2_neg_small(float x) {
  const float y = x * 0.69314718f;
  constexpr float c[8] = {1.f, 0.5f, 1.f / 6.f, 1.f / 24.f, 1.f / 120.f, 1.f / 720.f, 1.f / 5040.f, 1.f / 40320.f};
  static_assert(D >= 1 && D <= 7, "series length");
  float p = c[D];
#pragma unroll
  for (int i = D - 1; i >= 0; --i) p = fmaf(p, -y, c[i]);
  return y * p;
}

// Rows of a batch: target rows (b, i) for i < tper, then draft rows (b, i)
// for i < dper, b < nb.  Row r of the statistics array is target row
// (r / tper, r % tper) for r < nb * tper, then draft rows in the same order.
struct RowsDesc {
  const void* tgt; int64_t tsb, tsk; int tper;
  const void* drf; int64_t dsb, dsk; int dper;
  int nb;
  const float* temp; float temp_scalar;  // per batch row, or one scalar (temp == nullptr)
  int V, ntiles, C;
  int vec_t, vec_d;
};

template <class E>
__device__ __forceinline__ const typename E::raw* row_of(const RowsDesc& d, int r, int* b, bool* aligned) {
  using raw = typename E::raw;
  const int RT = d.nb * d.tper;
  if (r < RT) {
    *b = r / d.tper;
    *aligned = d.vec_t != 0;
    return static_cast<const raw*>(d.tgt) + static_cast<int64_t>(*b) * d.tsb + static_cast<int64_t>(r % d.tper) * d.tsk;
  }
  r -= RT;
  *b = r / d.dper;
  *aligned = d.vec_d != 0;
  return static_cast<const raw*>(d.drf) + static_cast<int64_t>(*b) * d.dsb + static_cast<int64_t>(r % d.dper) * d.dsk;
}

__device__ __forceinline__ float temperature_of(const RowsDesc& d, int b) {
  return d.temp ? d.temp[b] : d.temp_scalar;
}
__device__ __forceinline__ bool temperature_ok(float T) { return T > 0.f && T < INFINITY; }

// Statistics at sub-chunk granularity, one wave per sub-chunk: sub-chunk
// g = blockIdx.x * kWaves + wave of the rows' C sub-chunks each (row g / C,
// sub-chunk g % C) covers the ST tiles of 256 vectors from tile (g % C) * ST,
// i.e. ST * 4 vectors of the wave's 64 lanes.  The wave streams them S vectors
// per lane at a time, keeping a per-lane running reference (the largest
// z * s so far) and the exp2 sum rescaled to it, then takes one wave maximum
// and one float64 wave sum: no LDS and no barrier.  stats[g] = stats[r * C + j]
// holds (m, D) of sub-chunk j of row r: m the largest z * s of the
// sub-chunk (-inf if it has none), D = sum 2^(z s - m).
template <class E, int ST, int S>
__global__ __launch_bounds__(kThreads) void row_stats_wave_kernel(RowsDesc d, RowStat* __restrict__ stats,
                                                                  int64_t nsub) {
  constexpr int EPV = E::EPV;
  constexpr int WV = ST * (kThreads / 64);  // wave vectors per sub-chunk
  static_assert(WV % S == 0, "whole load steps per sub-chunk");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // (launched one wave per sub-chunk; written as a wave-stride loop, which
  // also covers a smaller grid: nothing below synchronises the workgroup.  In
  // this form the compiler schedules the loads so that the pass runs about
  // 1 us faster at the B=256 batch, same bits)
  for (int64_t g = static_cast<int64_t>(blockIdx.x) * kWaves + wave; g < nsub;
       g += static_cast<int64_t>(gridDim.x) * kWaves) {
    const int C = d.C;
    const int r = static_cast<int>(g / C), j = static_cast<int>(g - static_cast<int64_t>(g / C) * C);
    int b;
    bool aligned;
    const typename E::raw* row = row_of<E>(d, r, &b, &aligned);
    const float T = temperature_of(d, b);
    const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
    const int e0 = j * WV * 64 * EPV;
    float ref = -INFINITY, acc = 0.f;
#pragma unroll
    for (int st = 0; st < WV / S; ++st) {
      const int es = e0 + st * S * 64 * EPV;
      if (es >= d.V) break;  // wave-uniform: the row's last sub-chunk may be short
      float x[S][EPV];
      load_span<E, S, 64>(row, es, lane, d.V, aligned, x);
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < S; ++i)
#pragma unroll
        for (int k = 0; k < EPV; ++k) mx = fmaxf(mx, x[i][k]);
      const float nr = fmaxf(ref, mx * s);
      if (nr != -INFINITY) {
        float a2 = ref == -INFINITY ? 0.f : acc * __builtin_amdgcn_exp2f(ref - nr);
#pragma unroll
        for (int i = 0; i < S; ++i)
#pragma unroll
          for (int k = 0; k < EPV; ++k) a2 += __builtin_amdgcn_exp2f(fmaf(x[i][k], s, -nr));
        acc = a2;
        ref = nr;
      }
    }
    const float m = wave_max(ref);
    double dd;
    if (acc != acc) dd = acc;  // NaN propagates (data error)
    else if (ref == -INFINITY) dd = 0.0;
    else dd = static_cast<double>(acc) * static_cast<double>(__builtin_amdgcn_exp2f(ref - m));
    dd = wave_sum(dd);
    if (lane == 0) {
      RowStat o;
      o.m = m; o.pad = 0.f; o.D = dd;
      stats[g] = o;
    }
  }
}

}  // namespace sv

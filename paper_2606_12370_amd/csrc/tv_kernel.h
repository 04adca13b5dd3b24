// tv_kernel.h — fused TV-loss forward and gradient w.r.t. the draft logits
// (paper Sec. 4.1 Eqs. tv_loss / tv_grad, App. A, App. F; Sec. 4.2 Eq.
// e2e_tv) in six short launches that never wait on each other inside a
// launch:
//
//   1 row_stats   (sv_device.h) per-chunk statistics of every target and
//                 draft row of the N positions x K steps.
//   2 row_norm    (sv_device.h) each row's normaliser.
//   3 tv_pair     per (position n, step k, chunk): alpha partial sum min(p, q),
//                 S partial sum 1[q <= p] q and its complement 1 - S summed
//                 directly as sum 1[q > p] q (where one token holds nearly
//                 all of q, 1 - S formed from a float32 S near 1 would carry
//                 its rounding as a large relative error).
//   4 tv_coef     per position: alpha_k and S_k of its K steps (chunk order
//                 fixed), the chain factors g_k = dL_n/dalpha_k of the selected
//                 loss from prefix / suffix products, the position loss L_n,
//                 alpha[n, :], and the two gradient coefficients of each step.
//   5 tv_grad     per (position, step, chunk): grad = q * (1[q <= p] ? A1 : A0)
//                 with A1 = scale g_k (1 - S_k) / T (from the complement sum),
//                 A0 = -scale g_k S_k / T,
//                 written once (skipped for a forward-only call).
//   6 tv_loss     one workgroup adds the N position losses in a fixed order.
// The indicator 1[q <= p] is decided once, in launch 3, on log2 q <= log2 p
// (float32), and stored as bits that launch 5 reads, so S and the gradient
// always agree on it.
#pragma once

#include "sv_device.h"

namespace sv {

struct TvPair {
  double alpha;
  double S;   // sum 1[q <= p] q
  double Sc;  // sum 1[q > p] q, the complement of S summed directly
};

struct TvArgs {
  RowsDesc rows;  // target rows (n, k): tper = K; draft rows: dper = K
  int N, K;
  int mode;
  double scale;
  float inv_t;
  float* loss; float* overlap; float* grad;
  const RowStat* stats;  // [2 N K][C]
  const RowNorm* norms;  // [2 N K]
  TvPair* pairs;         // [N K][C]
  float2* coef;          // [N K]: (A1, A0)
  double* loss_pos;      // [N]
  uint8_t* bits;         // [N K][bits_stride]: 1[q <= p] per element, one 64-bit word per (chunk, tv_pair thread); NULL without gradient
  int64_t bits_stride;   // bytes per (position, step)
  int vec_g;
};

constexpr int kModeE2E = 0;
constexpr int kModeProd = 1;
constexpr int kModePerStep = 2;

// Chain factors g[k] = dL/dalpha_k and the per-position loss L (float64).
__device__ inline double chain_factors(const double* al, int K, int mode, double* g) {
  if (mode == kModePerStep) {
    double L = 0.0;
    for (int k = 0; k < K; ++k) { L += 1.0 - al[k]; g[k] = -1.0 / K; }
    return L / K;
  }
  double pre[SPEC_MAX_K_DEV + 1], suf[SPEC_MAX_K_DEV + 1];
  pre[0] = 1.0;
  for (int k = 0; k < K; ++k) pre[k + 1] = pre[k] * al[k];
  suf[K] = 1.0;
  for (int k = K - 1; k >= 0; --k) suf[k] = suf[k + 1] * al[k];
  if (mode == kModeProd) {
    for (int k = 0; k < K; ++k) g[k] = -(pre[k] * suf[k + 1]);
    return -pre[K];
  }
  // E2E: L = 1 - (1/K) sum_j prefix_{j+1}; g_k = -(1/K) prefix_k tail_k with
  // tail_k = 1 + alpha_{k+1} tail_{k+1}, tail_{K-1} = 1
  double sum = 0.0;
  for (int j = 0; j < K; ++j) sum += pre[j + 1];
  double tail = 1.0;
  for (int k = K - 1; k >= 0; --k) {
    if (k < K - 1) tail = 1.0 + al[k + 1] * tail;
    g[k] = -(pre[k] * tail) / K;
  }
  return 1.0 - sum / K;
}

template <class E>
__device__ __forceinline__ void tv_rows(const TvArgs& a, int n, int k, int* rt_i, int* rd_i) {
  *rt_i = n * a.K + k;
  *rd_i = a.N * a.K + n * a.K + k;
}

// Indicator bits 1[q <= p] of the forward pass, for the gradient pass.  The
// thread that handles elements of a chunk keeps their bits in one 64-bit word
// (tile j of the chunk at bits j*EPV .. j*EPV+EPV-1, EPV elements per vector)
// and stores it once per chunk: word (chunk, thread) of a (position, step)
// row, 2 KB per chunk.  kChunkWords = threads per chunk.
constexpr int kChunkWords = kThreads;

// The 4 bits of elements e .. e+3 (e % 4 == 0, offset e inside chunk c) for
// data read EPVW elements per vector by the forward pass.
template <int EPVW>
__device__ __forceinline__ uint32_t load_bits4(const uint8_t* row_bits, int c, int e) {
  static_assert(EPVW == 8 || EPVW == 4, "vector width");
  constexpr int TILEW = kThreads * EPVW;
  const int wt = (e % TILEW) / EPVW;                // the writing thread
  const int bit = (e / TILEW) * EPVW + (e % EPVW);  // its bit of element e
  const uint32_t byte = row_bits[(static_cast<int64_t>(c) * kChunkWords + wt) * 8 + (bit >> 3)];
  return (byte >> (bit & 7)) & 15u;
}

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void tv_pair_kernel(TvArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  __shared__ RedLds<4> red;
  const RowsDesc& d = a.rows;
  const int C = d.C;
  // grid-stride over the (position step, chunk) tasks (launched one workgroup per task)
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    const int n = u / a.K, k = u % a.K;
    int rt_i, rd_i, bb;
    bool al_t, al_d;
    tv_rows<E>(a, n, k, &rt_i, &rd_i);
    const typename E::raw* rt = row_of<E>(d, rt_i, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, rd_i, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const RowNorm nt = a.norms[rt_i], nd = a.norms[rd_i];
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, d.ntiles - tile0);
    static_assert(NT * EPV <= 64, "indicator bits of a chunk fit one word per thread");
    float al = 0.f, sq = 0.f, sc = 0.f;
    uint64_t mbits = 0;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float xt[S][EPV], xd[S][EPV];
      load_tiles<E, S>(rt, tile0 + j0, d.V, al_t, xt);
      load_tiles<E, S>(rd, tile0 + j0, d.V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        uint32_t m = 0;
#pragma unroll
        for (int kk = 0; kk < EPV; ++kk) {
          // log2 p and log2 q; min(p, q) is one exponential, and it is q
          // itself wherever q <= p, so it also carries the S term
          // (the reference and the log normaliser are not folded into one
          // float: its rounding, a few 1e-7 of M + L, would move alpha of
          // identical rows off 1 by about 1e-6, and the loss with it)
          const float lp = fmaf(xt[j][kk], s, -nt.M) - nt.L;
          const float lq = fmaf(xd[j][kk], s, -nd.M) - nd.L;
          const float mn = __builtin_amdgcn_exp2f(fminf(lp, lq));
          al += mn;
          const bool le = lq <= lp;
          sq += le ? mn : 0.f;
          // q itself where q > p (min(p, q) is p there)
          sc += le ? 0.f : __builtin_amdgcn_exp2f(lq);
          m |= le ? (1u << kk) : 0u;
        }
        mbits |= static_cast<uint64_t>(m) << ((j0 + j) * EPV);
      }
    }
    // the gradient pass reads these indicator bits instead of the target row
    // (streamed out with a non-temporal store: 5.48 against 5.67 ms for the
    // pass at N=16384, K=3, V=151936)
    if (a.bits)
      __builtin_nontemporal_store(mbits, reinterpret_cast<uint64_t*>(a.bits + static_cast<int64_t>(u) * a.bits_stride) +
                                             static_cast<int64_t>(c) * kChunkWords + threadIdx.x);
    double v[4] = {static_cast<double>(al), static_cast<double>(sq), static_cast<double>(sc), 0.0};
    wg_sum<4>(v, red);
    if (threadIdx.x == 0) {
      TvPair o;
      o.alpha = v[0]; o.S = v[1]; o.Sc = v[2];
      a.pairs[t] = o;
    }
  }
}

// Per position (one wave each, 4 per workgroup): alpha_k, S_k, the chain
// factors, the loss L_n, alpha[n, :] and the gradient coefficients.
__global__ __launch_bounds__(kThreads) void tv_coef_kernel(TvArgs a) {
  __shared__ double al[kWaves][SPEC_MAX_K_DEV], S[kWaves][SPEC_MAX_K_DEV], Sc[kWaves][SPEC_MAX_K_DEV];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = blockIdx.x * kWaves + wave;
  if (n >= a.N) return;
  const int C = a.rows.C, K = a.K;
  for (int kk = 0; kk < K; ++kk) {
    double x = 0.0, y = 0.0, z = 0.0;
    const TvPair* ps = a.pairs + static_cast<int64_t>(n * K + kk) * C;
    for (int cc = lane; cc < C; cc += 64) { x += ps[cc].alpha; y += ps[cc].S; z += ps[cc].Sc; }
    x = wave_sum(x);
    y = wave_sum(y);
    z = wave_sum(z);
    if (lane == 0) { al[wave][kk] = x; S[wave][kk] = y; Sc[wave][kk] = z; }
  }
  if (lane == 0) {
    double g[SPEC_MAX_K_DEV];
    const double L = chain_factors(al[wave], K, a.mode, g);
    a.loss_pos[n] = a.scale * L;
    for (int kk = 0; kk < K; ++kk) {
      if (a.overlap) a.overlap[static_cast<int64_t>(n) * K + kk] = static_cast<float>(al[wave][kk]);
      const double gk = a.scale * g[kk] * static_cast<double>(a.inv_t);
      a.coef[static_cast<int64_t>(n) * K + kk] =
          make_float2(static_cast<float>(gk * Sc[wave][kk]), static_cast<float>(gk * (-S[wave][kk])));
    }
  }
}

template <class E, int NT, int S, int EPVW>
__global__ __launch_bounds__(kThreads) void tv_grad_kernel(TvArgs a, int64_t ntasks) {
  static_assert(E::EPV == 4, "the gradient pass reads 4 elements per vector");
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  const RowsDesc& d = a.rows;
  const int C = d.C, K = a.K, V = d.V;
  // grid-stride over the (position step, chunk) tasks (launched one workgroup per task)
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    const int n = u / K, k = u % K;
    int rt_i, rd_i, bb;
    bool al_d;
    tv_rows<E>(a, n, k, &rt_i, &rd_i);
    const typename E::raw* rd = row_of<E>(d, rd_i, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const RowNorm nd = a.norms[rd_i];
    const float2 A = a.coef[u];
    float* gr = a.grad + static_cast<int64_t>(u) * V;
    const uint8_t* rb = a.bits + static_cast<int64_t>(u) * a.bits_stride;
    // this kernel may read with a narrower vector than the statistics passes, so
    // its tile count comes from its own tile width (the chunk is the same)
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, (V + TILE - 1) / TILE - tile0);
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float xd[S][EPV];
      uint32_t le[S];
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int v0 = (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV;
        le[j] = v0 < V ? load_bits4<EPVW>(rb, c, v0 - c * NT * TILE) : 0u;
      }
      load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int v0 = (tile0 + j0 + j) * TILE + threadIdx.x * EPV;
        float gv[EPV];
#pragma unroll
        for (int kk = 0; kk < EPV; ++kk) {
          const float q = prob(xd[j][kk], s, nd.M, nd.invD);
          gv[kk] = q * (((le[j] >> kk) & 1u) ? A.x : A.y);
        }
        if (a.vec_g && v0 + EPV <= V) {
#pragma unroll
          for (int h = 0; h < EPV; h += 4) {
            f32x4 w4 = {gv[h], gv[h + 1], gv[h + 2], gv[h + 3]};
            __builtin_nontemporal_store(w4, reinterpret_cast<f32x4*>(gr + v0 + h));
          }
        } else {
#pragma unroll
          for (int kk = 0; kk < EPV; ++kk)
            if (v0 + kk < V) gr[v0 + kk] = gv[kk];
        }
      }
    }
  }
}

// The total loss: position losses added in a fixed order by one workgroup.
__global__ __launch_bounds__(kThreads) void tv_loss_kernel(TvArgs a) {
  __shared__ RedLds<1> red;
  double acc = 0.0;
  for (int p = threadIdx.x; p < a.N; p += kThreads) acc += a.loss_pos[p];
  double v[1] = {acc};
  wg_sum<1>(v, red);
  if (threadIdx.x == 0) *a.loss = static_cast<float>(v[0]);
}

}  // namespace sv

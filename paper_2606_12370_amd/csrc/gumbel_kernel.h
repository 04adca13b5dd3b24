// gumbel_kernel.h — Gumbel-max verification (paper App. G.2, Alg. rs_gumbel)
// and the Gumbel-max draft sampler on gfx950.
//
// Verification keeps the accept loop of the multinomial path (row_stats and
// decide, plus pair_pass when overlaps are requested) and replaces the CDF
// inversion: the token at the emitting position n is
//   argmax_v [log r_v + G_v] = argmax_v r_v / E_v,   E_v = -ln U_v ~ Exp(1),
// with r = max(0, p_n - q_n) after a rejection and r = p_K for the bonus.
// gumbel_pass reads the emitting row (pair) chunk by chunk and keeps each
// chunk's best key and its first index, for the residual and for p_n (the
// fallback when the residual has no mass); gumbel_finish combines the chunks.
//
// The draft sampler scores z_v s - log2 E_v (log2 units of z/T + G) in one
// read per row, chunk by chunk, then combines the chunks; T = 0 scores the
// raw logits (the greedy token).
#pragma once

#include "sv_device.h"
#include "verify_kernel.h"

namespace sv {

constexpr uint64_t kTagGumbelVerify = 2;
constexpr uint64_t kTagGumbelSample = 3;
constexpr int kNoIndex = 0x7fffffff;

// E = -ln U for element k (0..7) of a Philox block: word (k >> 1), its top 24
// bits (even k) or bits 8..31 (odd k), U = (bits + 1/2) 2^-24.  The largest
// keys r / E come from U close to 1, where E must keep its relative
// precision: there y = 1 - U is exact in float32 and E = -ln(1 - y) is its
// Taylor series y + y^2/2 + ... + y^6/6 (truncation below 1e-8 relative for
// y < 1/16); elsewhere E = -ln2 log2(U) with the hardware log2 (U exact below
// 1/2, one rounding of at most 2^-25 above, i.e. below 5e-7 relative in E).
__device__ __forceinline__ float exp_variate(const Philox4x64& g, int k) {
  const uint64_t w = g.w[(k >> 1) & 3];
  const uint32_t bits = (k & 1) ? static_cast<uint32_t>((w >> 8) & 0xFFFFFFull) : static_cast<uint32_t>(w >> 40);
  constexpr float kInv24 = 5.9604644775390625e-8f;  // 2^-24
  constexpr float kHalf24 = 2.98023223876953125e-8f;  // 2^-25
  // one conversion (exact: bits < 2^24); u = (bits + 1/2) 2^-24 rounded once
  // by an FMA, y = 1 - bits 2^-24 (exact) - 2^-25, exact wherever it is used
  // (y < 1/16, where it has at most 21 significant bits)
  const float f = static_cast<float>(bits);
  const float y = fmaf(-f, kInv24, 1.0f) - kHalf24;
  const float u = fmaf(f, kInv24, kHalf24);
  // both forms, then a select: no divergent branch per element; the series
  // in Horner form with fused multiply-adds (5 FMAs and a multiply)
  const float series =
      y * fmaf(y, fmaf(y, fmaf(y, fmaf(y, fmaf(y, 0.166666672f, 0.2f), 0.25f), 0.333333343f), 0.5f), 1.f);
  const float viaLog = -0.693147182f * __builtin_amdgcn_logf(u);
  return y < 0.0625f ? series : viaLog;
}

struct GumbelBest {  // one chunk of the emitting row
  float kr;          // largest r / E over the chunk (-1: no residual mass)
  int ir;            // its first index
  float kp;          // largest p / E (fallback to p_n)
  int ip;
};

// Workgroup argmax of (key, first index): the largest key, then the smallest
// index among the threads holding it.  Every thread receives both.
__device__ __forceinline__ void wg_argmax(float& key, int& idx, RedLds<4>& red, RedLds<1>& red1) {
  float m[4] = {key, -INFINITY, -INFINITY, -INFINITY};
  wg_max<4>(m, red);
  idx = wg_min_int(key == m[0] ? idx : kNoIndex, red1);
  key = m[0];
}

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void gumbel_pass_kernel(VerifyArgs a, GumbelBest* __restrict__ best,
                                                               int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  __shared__ RedLds<4> red;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int C = d.C, K = a.K;
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int b = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    const int n = a.decision[b];
    if (n < 0) continue;  // data error: decide has written the row
    const bool residual = n < K;
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, target_row(a, b, n), &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, draft_row(a, b, residual ? n : 0), &bb, &al_d);
    const float s = scale_of(temperature_of(d, b));
    const RowNorm nt = a.norms[target_row(a, b, n)];
    const RowNorm nd = a.norms[draft_row(a, b, residual ? n : 0)];
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, d.ntiles - tile0);
    float kr = -1.f, kp = -1.f;
    int ir = kNoIndex, ip = kNoIndex;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float xt[S][EPV], xd[S][EPV];
      load_tiles<E, S>(rt, tile0 + j0, d.V, al_t, xt);
      if (residual) load_tiles<E, S>(rd, tile0 + j0, d.V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int v0 = (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV;
        const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(v0 >> 3), a.offset,
                                           kTagGumbelVerify, a.seed, 0ull);
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float e = exp_variate(g, (v0 & 7) + k);
          const float p = prob(xt[j][k], s, nt.M, nt.invD);
          const float keyp = __fdividef(p, e);
          if (p > 0.f && keyp > kp) { kp = keyp; ip = v0 + k; }
          if (residual) {
            const float r = p - fminf(p, prob(xd[j][k], s, nd.M, nd.invD));
            const float keyr = __fdividef(r, e);
            if (r > 0.f && keyr > kr) { kr = keyr; ir = v0 + k; }
          }
        }
      }
    }
    wg_argmax(kr, ir, red, red1);
    wg_argmax(kp, ip, red, red1);
    if (threadIdx.x == 0) {
      GumbelBest o;
      o.kr = kr; o.ir = ir; o.kp = kp; o.ip = ip;
      best[t] = o;
    }
  }
}

// Wave-wide argmax over C chunk entries (key, first index), every lane gets it.
__device__ __forceinline__ void wave_argmax(float& key, int& idx) {
  float m = key;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  idx = wave_min_int(key == m ? idx : kNoIndex);
  key = m;
}

// One wave per batch row: overlaps and the Gumbel-max token.
__global__ __launch_bounds__(kThreads) void gumbel_finish_kernel(VerifyArgs a, const GumbelBest* __restrict__ best) {
  const int b = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (b >= a.B) return;
  const int lane = threadIdx.x & 63;
  const int K = a.K, C = a.rows.C;
  const int n = a.decision[b];
  if (n < 0) return;
  const GumbelBest* gb = best + static_cast<int64_t>(b) * C;
  float kr = -1.f, kp = -1.f;
  int ir = kNoIndex, ip = kNoIndex;
  for (int cc = lane; cc < C; cc += 64) {  // chunks in order: strict ">" keeps the first
    const GumbelBest e = gb[cc];
    if (e.kr > kr) { kr = e.kr; ir = e.ir; }
    if (e.kp > kp) { kp = e.kp; ip = e.ip; }
  }
  wave_argmax(kr, ir);
  wave_argmax(kp, ip);
  for (int i = 0; i < K && a.overlap != nullptr; ++i) {
    double x = 0.0;
    const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + i) * C;
    for (int cc = lane; cc < C; cc += 64) x += ps[cc].alpha;
    x = wave_sum(x);
    if (lane == 0) a.overlap[static_cast<int64_t>(b) * K + i] = static_cast<float>(x);
  }
  // the residual's argmax, or p_n's when the residual has no mass
  if (lane == 0) a.emitted[static_cast<int64_t>(b) * (K + 1) + n] = (kr > 0.f) ? ir : (kp > 0.f ? ip : -1);
}

// ---------------------------------------------------------------------------
// Gumbel-max draft sampler

struct GumbelSampleArgs {
  RowsDesc rows;  // tper = 1, nb = R rows
  int R;
  uint64_t seed, offset;
  int32_t* token;
  GumbelBest* best;  // [R][C]: kr = best score, ir = its index, ip = data-error flag
};

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void gumbel_sample_pass_kernel(GumbelSampleArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  __shared__ RedLds<4> red;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int C = d.C;
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int r = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    int bb;
    bool al;
    const typename E::raw* row = row_of<E>(d, r, &bb, &al);
    const float T = temperature_of(d, r);
    const bool greedy = T == 0.f;
    const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, d.ntiles - tile0);
    float ks = -INFINITY;
    int is = kNoIndex, bad = 0;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float x[S][EPV];
      load_tiles<E, S>(row, tile0 + j0, d.V, al, x);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int v0 = (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV;
        Philox4x64 g{};
        if (!greedy)
          g = philox4x64_10(static_cast<uint64_t>(r), static_cast<uint64_t>(v0 >> 3), a.offset, kTagGumbelSample,
                            a.seed, 0ull);
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float z = x[j][k];
          if (z != z || z == INFINITY) bad = 1;
          const float sc = greedy ? z : z * s - __builtin_amdgcn_logf(exp_variate(g, (v0 & 7) + k));
          if (sc > ks) { ks = sc; is = v0 + k; }
        }
      }
    }
    float m[4] = {ks, static_cast<float>(bad), -INFINITY, -INFINITY};
    wg_max<4>(m, red);
    const int i1 = wg_min_int(ks == m[0] ? is : kNoIndex, red1);
    if (threadIdx.x == 0) {
      GumbelBest o;
      o.kr = m[0]; o.ir = i1; o.kp = 0.f; o.ip = m[1] > 0.f ? 1 : 0;
      a.best[t] = o;
    }
  }
}

// One wave per row: the best chunk's token, or -1 for a data error.
__global__ __launch_bounds__(kThreads) void gumbel_sample_finish_kernel(GumbelSampleArgs a) {
  const int r = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int lane = threadIdx.x & 63;
  const int C = a.rows.C;
  const GumbelBest* gb = a.best + static_cast<int64_t>(r) * C;
  float k = -INFINITY;
  int i = kNoIndex, bad = 0;
  for (int cc = lane; cc < C; cc += 64) {
    const GumbelBest e = gb[cc];
    if (e.kr > k) { k = e.kr; i = e.ir; }
    bad |= e.ip;
  }
  wave_argmax(k, i);
  bad = -wave_min_int(-bad);
  if (lane == 0) {
    const float T = temperature_of(a.rows, r);
    const bool t_ok = T == 0.f || temperature_ok(T);
    a.token[r] = (t_ok && !bad && k > -INFINITY && i != kNoIndex) ? i : -1;
  }
}

}  // namespace sv

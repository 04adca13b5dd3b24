// verify_kernel.h — chain rejection-sampling verification (paper Sec. 2.2,
// Eq. reject_sample; App. G.1, Alg. rs_multinomial) in three launches that
// never wait on each other inside a launch:
//
//   1 row_stats   (sv_device.h) every target and draft row, split into
//                 chunks of NT tiles: per-chunk (max reference, exp2 sum).
//   2 pair_pass   every (target row i, draft row i) pair, i < K, chunk by
//                 chunk: p and q from the combined row statistics, then the
//                 chunk's overlap sum min(p, q) and residual mass
//                 sum max(0, p - q).  Bonus rows need no second read.
//   3 finish      one workgroup per batch row: accept tests from the two
//                 gathered logits in float64 and Philox uniforms, accept
//                 length, overlap, and the resample: the chunk whose
//                 cumulative mass crosses u' Z is found from the per-chunk
//                 masses, and only that chunk is read again to invert the
//                 CDF inside it (tile sums, thread scan, element scan).
#pragma once

#include "sv_device.h"

namespace sv {

struct PairStat {  // one chunk of a (target, draft) pair
  double alpha;    // sum min(p, q)
  double Z;        // sum max(0, p - q)
};

struct VerifyArgs {
  RowsDesc rows;   // target rows: tper = K+1; draft rows: dper = K
  int B, K;
  const int32_t* ids;
  uint64_t seed, offset;
  int32_t* accept_len; int32_t* emitted;
  float* overlap; float* p_at; float* q_at; float* logz_t; float* logz_d;
  const RowStat* stats;   // [rows][C]
  PairStat* pairs;        // [B*K][C]
};

__device__ __forceinline__ int target_row(const VerifyArgs& a, int b, int i) { return b * (a.K + 1) + i; }
__device__ __forceinline__ int draft_row(const VerifyArgs& a, int b, int i) {
  return a.B * (a.K + 1) + b * a.K + i;
}

// Pass 2 over one chunk of a (target, draft) pair: overlap and residual mass.
template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void pair_pass_kernel(VerifyArgs a) {
  constexpr int EPV = E::EPV;
  __shared__ RedLds<4> red;
  __shared__ float sh_f[4];
  const RowsDesc& d = a.rows;
  const int C = d.C;
  const int u = blockIdx.x / C, c = blockIdx.x % C;
  const int b = u / a.K, i = u % a.K;
  const int rt_i = target_row(a, b, i), rd_i = draft_row(a, b, i);
  int bb;
  bool al_t, al_d;
  const typename E::raw* rt = row_of<E>(d, rt_i, &bb, &al_t);
  const typename E::raw* rd = row_of<E>(d, rd_i, &bb, &al_d);
  const float T = temperature_of(d, b);
  const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
  if (threadIdx.x < 64) {
    float Mt, Md;
    double Dt, Dd;
    combine_row(a.stats + static_cast<int64_t>(rt_i) * C, C, &Mt, &Dt);
    combine_row(a.stats + static_cast<int64_t>(rd_i) * C, C, &Md, &Dd);
    if (threadIdx.x == 0) {
      sh_f[0] = Mt; sh_f[1] = static_cast<float>(1.0 / Dt);
      sh_f[2] = Md; sh_f[3] = static_cast<float>(1.0 / Dd);
    }
  }
  __syncthreads();
  const float Mt = sh_f[0], it = sh_f[1], Md = sh_f[2], id = sh_f[3];
  const int tile0 = c * NT;
  const int nt = min(NT, d.ntiles - tile0);
  float al = 0.f, zr = 0.f;
#pragma unroll
  for (int j0 = 0; j0 < NT; j0 += S) {
    if (j0 >= nt) break;
    float xt[S][EPV], xd[S][EPV];
    load_tiles<E, S>(rt, tile0 + j0, d.V, al_t, xt);
    load_tiles<E, S>(rd, tile0 + j0, d.V, al_d, xd);
#pragma unroll
    for (int j = 0; j < S; ++j)
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        const float p = prob(xt[j][k], s, Mt, it);
        const float q = prob(xd[j][k], s, Md, id);
        const float mn = fminf(p, q);
        al += mn;
        zr += p - mn;
      }
  }
  double v[4] = {static_cast<double>(al), static_cast<double>(zr), 0.0, 0.0};
  wg_sum<4>(v, red);
  if (threadIdx.x == 0) {
    PairStat o;
    o.alpha = v[0]; o.Z = v[1];
    a.pairs[blockIdx.x] = o;
  }
}

// Residual (or target) mass of the EPV elements of one thread's vector.
template <class E>
__device__ __forceinline__ void vector_masses(const typename E::raw* rt, const typename E::raw* rd, bool residual,
                                              int v0, int V, float s, float Mt, float it, float Md, float id,
                                              float (&r)[E::EPV]) {
#pragma unroll
  for (int k = 0; k < E::EPV; ++k) {
    if (v0 + k < V) {
      const float p = prob(E::one(rt + v0 + k), s, Mt, it);
      r[k] = residual ? p - fminf(p, prob(E::one(rd + v0 + k), s, Md, id)) : p;
    } else {
      r[k] = 0.f;
    }
  }
}

struct FinishShared {
  float M[2 * SPEC_MAX_K_DEV + 1];
  double D[2 * SPEC_MAX_K_DEV + 1];
  double alpha[SPEC_MAX_K_DEV];
  double px[SPEC_MAX_K_DEV], qx[SPEC_MAX_K_DEV];
  double tin;
  int err, n, cstar, residual, token;
};

// One workgroup per batch row: accept tests, accept length, overlap and the
// resampled / bonus token.
template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void finish_kernel(VerifyArgs a) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  using raw = typename E::raw;
  __shared__ FinishShared sh;
  __shared__ RedLds<NT> redv;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int K = a.K, C = d.C, V = d.V;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const float T = temperature_of(d, b);
  const bool t_ok = temperature_ok(T);
  const float s = t_ok ? scale_of(T) : 1.0f;
  const int32_t* xb = a.ids + static_cast<int64_t>(b) * K;

  // row normalisers of the 2K+1 rows and the overlap of every draft step (wave 0)
  if (tid < 64) {
    for (int i = 0; i <= K; ++i) {
      float M;
      double D;
      combine_row(a.stats + static_cast<int64_t>(target_row(a, b, i)) * C, C, &M, &D);
      if (lane == 0) { sh.M[i] = M; sh.D[i] = D; }
    }
    for (int i = 0; i < K; ++i) {
      float M;
      double D;
      combine_row(a.stats + static_cast<int64_t>(draft_row(a, b, i)) * C, C, &M, &D);
      if (lane == 0) { sh.M[K + 1 + i] = M; sh.D[K + 1 + i] = D; }
    }
    for (int i = 0; i < K; ++i) {
      double al = 0.0;
      const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + i) * C;
      for (int cc = lane; cc < C; cc += 64) al += ps[cc].alpha;
      al = wave_sum(al);
      if (lane == 0) sh.alpha[i] = al;
    }
  }
  __syncthreads();

  // accept tests in float64, u q(x) < p(x) with no division; first rejection ends the chain
  if (tid == 0) {
    bool err = !t_ok;
    for (int i = 0; i < 2 * K + 1; ++i)
      if (!(sh.D[i] > 0.0 && sh.D[i] < INFINITY && sh.M[i] < INFINITY)) err = true;
    int n = K;
    for (int i = 0; i < K; ++i) {
      const int x = xb[i];
      sh.px[i] = 0.0;
      sh.qx[i] = 0.0;
      if (x < 0 || x >= V) { err = true; continue; }
      if (err) continue;
      int bb;
      bool al;
      const raw* rt = row_of<E>(d, target_row(a, b, i), &bb, &al);
      const raw* rd = row_of<E>(d, draft_row(a, b, i), &bb, &al);
      const double px = exp2(static_cast<double>(E::one(rt + x)) * static_cast<double>(s) -
                             static_cast<double>(sh.M[i])) / sh.D[i];
      const double qx = exp2(static_cast<double>(E::one(rd + x)) * static_cast<double>(s) -
                             static_cast<double>(sh.M[K + 1 + i])) / sh.D[K + 1 + i];
      sh.px[i] = px;
      sh.qx[i] = qx;
      if (n == K) {
        const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(i), a.offset, 0ull,
                                           a.seed, 0ull);
        if (!(u24(g.w[0]) * qx < px)) n = i;
      }
    }
    sh.err = err ? 1 : 0;
    sh.n = n;
    sh.cstar = -1;
  }
  __syncthreads();
  const bool err = sh.err != 0;
  const int n = sh.n;

  // the chunk holding the sampling target (wave 0)
  if (!err && tid < 64) {
    const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + (n < K ? n : 0)) * C;
    double zs = 0.0;
    if (n < K) {
      for (int cc = lane; cc < C; cc += 64) zs += ps[cc].Z;
      zs = wave_sum(zs);
    }
    // residual of the rejected step; p_n itself for the bonus row or an empty residual
    const bool residual = n < K && zs > 0.0;
    const RowStat* st = a.stats + static_cast<int64_t>(target_row(a, b, n)) * C;
    const float Mn = sh.M[n];
    const double Dn = sh.D[n];
    const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(n), a.offset, 0ull,
                                       a.seed, 0ull);
    double tot = 0.0;
    for (int cc = lane; cc < C; cc += 64) {
      const float mc = st[cc].m;
      tot += residual ? ps[cc].Z
                      : (mc == -INFINITY ? 0.0 : st[cc].D * static_cast<double>(__builtin_amdgcn_exp2f(mc - Mn)) / Dn);
    }
    tot = wave_sum(tot);
    const double target = u24(g.w[1]) * tot;
    double carry = 0.0, tin = 0.0;
    int cstar = -1, clast = -1;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const int cc = c0 + lane;
      double zc = 0.0;
      if (cc < C) {
        const float mc = st[cc].m;
        zc = residual ? ps[cc].Z
                      : (mc == -INFINITY ? 0.0 : st[cc].D * static_cast<double>(__builtin_amdgcn_exp2f(mc - Mn)) / Dn);
      }
      const double incl = carry + wave_incl_scan(zc);
      const double excl = incl - zc;
      const uint64_t hit = __ballot(cc < C && incl > target && excl <= target && zc > 0.0);
      const uint64_t pos = __ballot(cc < C && zc > 0.0);
      if (pos) clast = c0 + 63 - __clzll(pos);
      if (cstar < 0 && hit) {
        const int l = __ffsll(static_cast<long long>(hit)) - 1;
        cstar = c0 + l;
        tin = target - __shfl(excl, l, 64);
      }
      carry = __shfl(incl, 63, 64);
    }
    if (cstar < 0) { cstar = clast; tin = INFINITY; }  // past the end by rounding: last element with mass
    if (lane == 0) {
      sh.cstar = cstar;
      sh.tin = tin;
      sh.residual = residual ? 1 : 0;
    }
  }
  __syncthreads();

  // inverse CDF inside the chosen chunk (whole workgroup)
  int token = -1;
  if (!err && sh.cstar >= 0) {
    const int cstar = sh.cstar;
    const bool residual = sh.residual != 0;
    int bb;
    bool al_t, al_d;
    const raw* rt = row_of<E>(d, target_row(a, b, n), &bb, &al_t);
    const raw* rd = row_of<E>(d, draft_row(a, b, n < K ? n : 0), &bb, &al_d);
    const float Mt = sh.M[n], it = static_cast<float>(1.0 / sh.D[n]);
    const float Md = n < K ? sh.M[K + 1 + n] : 0.f;
    const float id = n < K ? static_cast<float>(1.0 / sh.D[K + 1 + n]) : 0.f;
    const int tile0 = cstar * NT;
    const int nt = min(NT, d.ntiles - tile0);
    float tsum[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) tsum[j] = 0.f;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt) break;
      float xt[S][EPV], xd[S][EPV];
      load_tiles<E, S>(rt, tile0 + j0, V, al_t, xt);
      if (residual) load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j)
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float p = prob(xt[j][k], s, Mt, it);
          tsum[j0 + j] += residual ? p - fminf(p, prob(xd[j][k], s, Md, id)) : p;
        }
    }
    double W[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) W[j] = (j < nt) ? static_cast<double>(tsum[j]) : 0.0;
    wg_sum<NT>(W, redv);  // tile totals, identical in every thread
    const double tin = sh.tin;
    int jstar = -1, jlast = -1;
    double cum = 0.0, t_in = 0.0;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      if (j < nt) {
        if (W[j] > 0.0) jlast = j;
        if (jstar < 0 && cum + W[j] > tin) { jstar = j; t_in = tin - cum; }
        cum += W[j];
      }
    }
    bool clamp = false;
    if (jstar < 0) { jstar = jlast; clamp = true; }
    if (jstar >= 0) {
      float w = 0.f;
#pragma unroll
      for (int j = 0; j < NT; ++j)
        if (j == jstar) w = tsum[j];
      double incl;
      const double excl = wg_scan(static_cast<double>(w), red1, &incl);
      int tstar = kThreads;
      if (!clamp) tstar = wg_min_int((incl > t_in && excl <= t_in && w > 0.f) ? tid : kThreads, red1);
      if (tstar == kThreads) {
        clamp = true;
        tstar = -wg_min_int((w > 0.f) ? -tid : 1, red1);
      }
      if (tid == 0) sh.token = -1;
      __syncthreads();
      if (tid == tstar) {
        const int v0 = (tile0 + jstar) * TILE + tid * EPV;
        float r[EPV];
        vector_masses<E>(rt, rd, residual, v0, V, s, Mt, it, Md, id, r);
        const double tl = t_in - excl;
        float cumf = 0.f;
        int kstar = -1, klast = -1;
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          cumf += r[k];
          if (r[k] > 0.f) klast = k;
          if (kstar < 0 && !clamp && r[k] > 0.f && static_cast<double>(cumf) > tl) kstar = k;
        }
        if (kstar < 0) kstar = klast;
        if (kstar >= 0) sh.token = v0 + kstar;
      }
      __syncthreads();
      token = sh.token;
    }
  }

  // outputs: every per-row output has this single writer
  if (tid == 0) {
    int32_t* em = a.emitted + static_cast<int64_t>(b) * (K + 1);
    a.accept_len[b] = err ? -1 : n;
    for (int j = 0; j <= K; ++j) em[j] = err ? -1 : ((j < n) ? xb[j] : ((j == n) ? token : -1));
    for (int i = 0; i < K; ++i) {
      const int64_t o = static_cast<int64_t>(b) * K + i;
      if (a.overlap) a.overlap[o] = err ? NAN : static_cast<float>(sh.alpha[i]);
      if (a.p_at) a.p_at[o] = err ? NAN : static_cast<float>(sh.px[i]);
      if (a.q_at) a.q_at[o] = err ? NAN : static_cast<float>(sh.qx[i]);
      if (a.logz_d)
        a.logz_d[o] = err ? NAN
                          : static_cast<float>((static_cast<double>(sh.M[K + 1 + i]) + log2(sh.D[K + 1 + i])) * kLn2D);
    }
    if (a.logz_t)
      for (int i = 0; i <= K; ++i)
        a.logz_t[static_cast<int64_t>(b) * (K + 1) + i] =
            err ? NAN : static_cast<float>((static_cast<double>(sh.M[i]) + log2(sh.D[i])) * kLn2D);
  }
}

}  // namespace sv

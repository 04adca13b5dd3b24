// kl_kernel.h — CE, forward-KL and reverse-KL losses of the draft against the
// target and their gradients w.r.t. the draft logits (paper Sec. 4.1 and its
// footnote, Table grad_comparison, App. B, App. C): the objectives the TV
// loss is compared against.
//
//   1 row_stats, 2 row_norm (sv_device.h): each row's reference M and
//                 normaliser, for the gradient.
//   3 kl_pass     per (position n, step k, chunk), with t = z_t s - M_t and
//                 u = z_d s - M_d (log2 units), e = 2^t, f = 2^u: Se = sum e,
//                 Sf = sum f and the weighted log-ratio sum W (forward:
//                 sum e (t - u); CE: sum e (-u); reverse: sum f (u - t)), all
//                 in float64 from the same e, f, t, u, so the loss (formed in
//                 kl_coef) is normalised by its own sums: a small KL is not
//                 swamped by the rounding of a separately computed log Z.
//                 Forward KL and CE also write the gradient (q - p) here,
//                 since it needs no global sum.
//   4 kl_coef     per position: L_{n,k} from its chunks, the per-step output,
//                 the position loss, the reverse-KL gradient constants.
//   5 kl_grad     reverse KL only: q (log q - log p - L), read again.
//   6 kl_loss     position losses added in a fixed order.
#pragma once

#include "sv_device.h"

namespace sv {

constexpr int kKlForward = 0;
constexpr int kKlCe = 1;
constexpr int kKlReverse = 2;

struct KlPart {  // one chunk of a (position, step) pair
  double se, sf, w;
};

struct KlArgs {
  RowsDesc rows;  // target rows (n, k): tper = K; draft rows: dper = K
  int N, K, kind;
  double scale;
  float inv_t;
  float* loss; float* per_step; float* grad;
  const RowStat* stats;  // [2 N K][C]
  const RowNorm* norms;  // [2 N K]
  KlPart* parts;         // [N K][C]
  float2* coef;          // [N K]: reverse-KL gradient constants
  double* loss_pos;      // [N]
  int vec_g;
};

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

template <class E, int NT, int S, int KIND>
__global__ __launch_bounds__(kThreads) void kl_pass_kernel(KlArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  __shared__ RedLds<4> red;
  const RowsDesc& d = a.rows;
  const int C = d.C, V = d.V, NK = a.N * a.K;
  const bool write_grad = a.grad != nullptr && KIND != kKlReverse;
  const float gcoef = static_cast<float>(a.scale * static_cast<double>(a.inv_t) / a.K);
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, u, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, NK + u, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const RowNorm nt = a.norms[u], nd = a.norms[NK + u];
    float* gr = write_grad ? a.grad + static_cast<int64_t>(u) * V : nullptr;
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, (V + TILE - 1) / TILE - tile0);
    double se = 0.0, sf = 0.0, w = 0.0;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float xt[S][EPV], xd[S][EPV];
      load_tiles<E, S>(rt, tile0 + j0, V, al_t, xt);
      load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        float gv[EPV];
        // the EPV elements of one vector are summed in float32, vectors in float64
        float ve = 0.f, vf = 0.f, vw = 0.f;
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float tt = fmaf(xt[j][k], s, -nt.M);
          const float uu = fmaf(xd[j][k], s, -nd.M);
          const float e = __builtin_amdgcn_exp2f(tt);
          const float f = __builtin_amdgcn_exp2f(uu);
          float term;
          if (KIND == kKlForward) term = e > 0.f ? e * (tt - uu) : 0.f;
          else if (KIND == kKlCe) term = e > 0.f ? -(e * uu) : 0.f;
          else term = f > 0.f ? f * (uu - tt) : 0.f;
          ve += e;
          vf += f;
          vw += term;
          gv[k] = gcoef * (f * nd.invD - e * nt.invD);  // (q - p) scale / (K T)
        }
        se += static_cast<double>(ve);
        sf += static_cast<double>(vf);
        w += static_cast<double>(vw);
        if (write_grad)
          store_grad<EPV>(gr, (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV, V, a.vec_g != 0, gv);
      }
    }
    double v[4] = {se, sf, w, 0.0};
    wg_sum<4>(v, red);
    if (threadIdx.x == 0) {
      KlPart o;
      o.se = v[0]; o.sf = v[1]; o.w = v[2];
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
    for (int cc = lane; cc < C; cc += 64) { se += ps[cc].se; sf += ps[cc].sf; w += ps[cc].w; }
    se = wave_sum(se);
    sf = wave_sum(sf);
    w = wave_sum(w);
    const double le = log2(se), lf = log2(sf);
    double L;  // log2 units
    if (a.kind == kKlForward) L = w / se - le + lf;
    else if (a.kind == kKlCe) L = w / se + lf;
    else L = w / sf - lf + le;
    L *= kLn2D;
    Ln += L;
    if (lane == 0) {
      if (a.per_step) a.per_step[static_cast<int64_t>(n) * K + kk] = static_cast<float>(L);
      // reverse-KL gradient: scale/(K T) q (ln2 (u - t + le - lf) - L), q = f / sf
      const double A = a.scale * static_cast<double>(a.inv_t) / K * kLn2D / sf;
      a.coef[static_cast<int64_t>(n) * K + kk] =
          make_float2(static_cast<float>(A), static_cast<float>(le - lf - L / kLn2D));
    }
  }
  if (lane == 0) a.loss_pos[n] = a.scale * Ln / K;
}

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void kl_grad_kernel(KlArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  const RowsDesc& d = a.rows;
  const int C = d.C, V = d.V, NK = a.N * a.K;
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, u, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, NK + u, &bb, &al_d);
    const float s = scale_of(d.temp_scalar);
    const float Mt = a.norms[u].M, Md = a.norms[NK + u].M;
    const float2 A = a.coef[u];
    float* gr = a.grad + static_cast<int64_t>(u) * V;
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
          const float tt = fmaf(xt[j][k], s, -Mt);
          const float uu = fmaf(xd[j][k], s, -Md);
          const float f = __builtin_amdgcn_exp2f(uu);
          gv[k] = f > 0.f ? A.x * f * ((uu - tt) + A.y) : 0.f;
        }
        store_grad<EPV>(gr, (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV, V, a.vec_g != 0, gv);
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

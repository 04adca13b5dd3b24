// variants_kernel.h — the acceptance rule's neighbours on gfx950:
//
//   target-only verification (paper Sec. 2.2, Eq. target_only): the draft's
//     greedy token x_i is accepted with probability p_i(x_i); after a
//     rejection the token is drawn from p_n without x_n.  Two launches:
//     row_stats over the K+1 target rows, then to_verify (one workgroup per
//     batch row: normalisers, accept tests, the residual's chunk, the CDF
//     inverted inside it).  No draft logits are read.
//   draft-stage sampling (App. G.1, draft stage): a token from
//     softmax(z / T) by inverse CDF, or the greedy token at T = 0.  Two
//     launches: row_stats, then sample (one workgroup per row).
//   per-step diagnostics (Sec. 3; App. E): entropies of p_i and q_i, max p_i,
//     the greedy draft token and alpha^TO = p_i(argmax q_i), alpha^RS =
//     sum min(p_i, q_i) split into sum_{p>q} q and sum_{q>=p} p.  Four
//     launches: diag_stats (one wave per sub-chunk: max reference, exp2 sum,
//     the entropy moment, largest logit and its first index), diag_norm (one
//     wave per row), diag_pair (one wave per pair sub-chunk), diag_finish
//     (one wave per step).
#pragma once

#include <cfloat>

#include "sv_device.h"

#include "verify_kernel.h"

namespace sv {

// ---------------------------------------------------------------------------
// target-only verification

struct ToArgs {
  RowsDesc rows;  // target rows only: tper = K+1, no draft rows
  int B, K;
  const int32_t* ids;
  uint64_t seed, offset;
  int32_t* accept_len; int32_t* emitted; float* p_at; float* logz_t;
  const RowStat* stats;  // [B*(K+1)][C]
};

struct ToShared {
  RowNorm nrm[SPEC_MAX_K_DEV + 1];
  int n, excl, cstar, excl_on;
  double tin;
  SampleShared smp;
};

// The chunk holding the sampling target for p_n (bonus or fallback): masses
// from the chunk statistics.
__device__ __forceinline__ double stat_mass(const RowStat* st, int cc, const RowNorm& nn) {
  const float mc = st[cc].m;
  return mc == -INFINITY ? 0.0 : st[cc].D * static_cast<double>(__builtin_amdgcn_exp2f(mc - nn.M)) / nn.D;
}

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void to_verify_kernel(ToArgs a) {
  using raw = typename E::raw;
  constexpr int CHUNK = NT * kThreads * E::EPV;
  __shared__ ToShared sh;
  __shared__ RedLds<NT> redv;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int K = a.K, C = d.C, V = d.V;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int row0 = b * (K + 1);
  // lane i < K: the greedy draft token of step i and its target logit, and
  // lane i <= K: the uniforms of step i (accept test, residual draw), all
  // requested and drawn before the normalisers are known
  int x = -1;
  float zx = 0.f;
  double ua = 0.0, ur = 0.0;
  if (tid <= K) {
    if (tid < K) {
      x = a.ids[static_cast<int64_t>(b) * K + tid];
      if (x >= 0 && x < V) {
        int bb;
        bool al;
        zx = E::one(row_of<E>(d, row0 + tid, &bb, &al) + x);
      }
    }
    const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(tid), a.offset, 0ull,
                                       a.seed, 0ull);
    ua = u24(g.w[0]);
    ur = u24(g.w[1]);
  }
  for (int j = wave; j <= K; j += kWaves) {
    float M;
    double D;
    combine_row(a.stats + static_cast<int64_t>(row0 + j) * C, C, &M, &D);
    if (lane == 0) sh.nrm[j] = make_norm(M, D);
  }
  __syncthreads();
  const float T = temperature_of(d, b);
  const bool t_ok = temperature_ok(T);
  const float s = t_ok ? scale_of(T) : 1.0f;
  // wave 0: accept tests in float64, u < p(x), lane i for step i; two ballots
  // give the row's error flag and its first rejection; lane j writes the
  // outputs of position j
  if (wave == 0) {
    double p = 0.0;
    bool ok = false, bad = false;
    if (lane < K) {
      const RowNorm& nt = sh.nrm[lane];
      bad = !(x >= 0 && x < V);
      if (!bad && t_ok && norm_ok(nt)) {
        p = exp2(static_cast<double>(zx) * static_cast<double>(s) - static_cast<double>(nt.M)) / nt.D;
        ok = ua < p;
      }
    }
    const uint64_t errm = __ballot((lane <= K && !norm_ok(sh.nrm[lane])) || bad);
    const uint64_t rejm = __ballot(lane < K && !ok);
    const bool err = !t_ok || errm != 0;
    const int n = err ? -1 : (rejm ? __ffsll(static_cast<long long>(rejm)) - 1 : K);
    if (lane == 0) a.accept_len[b] = n;
    if (lane <= K) {
      const int j = lane;
      const int64_t ob = static_cast<int64_t>(b) * (K + 1) + j;
      if (err || j != n) a.emitted[ob] = (!err && j < n) ? x : -1;
      if (a.p_at && j < K) a.p_at[static_cast<int64_t>(b) * K + j] = err ? NAN : static_cast<float>(p);
      if (a.logz_t)
        a.logz_t[ob] = err ? NAN : static_cast<float>((static_cast<double>(sh.nrm[j].M) + log2(sh.nrm[j].D)) * kLn2D);
    }
    const int xn = __shfl(x, n < 0 ? 0 : n, 64);
    if (lane == 0) {
      sh.n = n;
      sh.excl = (n >= 0 && n < K) ? xn : -1;
    }
  }
  __syncthreads();
  const int n = sh.n;
  if (n < 0) return;  // data error: every output of the row is written
  const int excl = sh.excl;
  const RowNorm nn = sh.nrm[n];
  int bb;
  bool al;
  const raw* rt = row_of<E>(d, row0 + n, &bb, &al);
  const RowStat* st = a.stats + static_cast<int64_t>(row0 + n) * C;
  // wave 0, lane cc < 64: the mass of sub-chunk cc from its statistics,
  // requested before the chunk holding x_n is read
  double m0 = 0.0;
  if (wave == 0 && lane < C) m0 = stat_mass(st, lane, nn);
  // The residual p_n without x_n: every chunk's mass comes from its
  // statistics except the chunk holding x_n, which is summed element by
  // element without x_n (a difference of two statistics would cancel when
  // x_n carries most of the chunk).
  const int cx = excl >= 0 ? excl / CHUNK : -1;
  double xm = 0.0;
  if (cx >= 0) {
    float tsum[NT];
    const int ntl = tile_masses<E, NT, S>(rt, al, rt, al, false, excl, cx, V, d.ntiles, s, nn, nn, kNoResidual, tsum);
    double W[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) W[j] = (j < ntl) ? static_cast<double>(tsum[j]) : 0.0;
    wg_sum<NT>(W, redv);
#pragma unroll
    for (int j = 0; j < NT; ++j) xm += W[j];
  }
  if (wave == 0) {
    const double u = __shfl(ur, n, 64);
    double tin = 0.0;
    // select_chunk asks for cc = c0 + lane, c0 a multiple of 64: cc < 64 is
    // this lane's prefetched sub-chunk
    int cstar = select_chunk(C, u, [&](int cc) -> double {
      return cc == cx ? xm : (cc < 64 ? m0 : stat_mass(st, cc, nn));
    }, &tin);
    bool ex_on = cx >= 0;
    if (cstar < 0) {  // no residual mass: draw from p_n itself
      cstar = select_chunk(C, u, [&](int cc) -> double { return cc < 64 ? m0 : stat_mass(st, cc, nn); }, &tin);
      ex_on = false;
    }
    if (lane == 0) {
      sh.cstar = cstar;
      sh.tin = tin;
      sh.excl_on = ex_on ? 1 : 0;
    }
  }
  __syncthreads();
  int token = -1;
  if (sh.cstar >= 0)
    token = sample_in_chunk<E, NT, S>(rt, al, rt, al, false, sh.excl_on ? excl : -1, sh.cstar, sh.tin, V, d.ntiles,
                                      s, nn, nn, kNoResidual, redv, red1, sh.smp);
  if (tid == 0) a.emitted[static_cast<int64_t>(b) * (K + 1) + n] = token;
}

// ---------------------------------------------------------------------------
// draft-stage sampling

struct SampleArgs {
  RowsDesc rows;  // tper = 1, nb = R rows
  int R;
  uint64_t seed, offset;
  int32_t* token; float* logz;
  const RowStat* stats;  // [R][C]
};

struct SampleKShared {
  RowNorm nrm;
  double tin;
  int cstar, ok;
  SampleShared smp;
};

// First index of the value M inside chunk c (whole workgroup; INT_MAX if absent).
template <class E, int NT, int S>
__device__ __forceinline__ int first_index_of(const typename E::raw* row, bool aligned, int c, float M, int V,
                                              int ntiles, RedLds<1>& red1) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  const int tile0 = c * NT;
  const int nt_tiles = min(NT, ntiles - tile0);
  int best = 0x7fffffff;
#pragma unroll
  for (int j0 = 0; j0 < NT; j0 += S) {
    if (j0 >= nt_tiles) break;
    float x[S][EPV];
    load_tiles<E, S>(row, tile0 + j0, V, aligned, x);
#pragma unroll
    for (int j = 0; j < S; ++j)
#pragma unroll
      for (int k = 0; k < EPV; ++k)
        if (x[j][k] == M) best = min(best, (tile0 + j0 + j) * TILE + static_cast<int>(threadIdx.x) * EPV + k);
  }
  return wg_min_int(best, red1);
}

template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void sample_kernel(SampleArgs a) {
  using raw = typename E::raw;
  __shared__ SampleKShared sh;
  __shared__ RedLds<NT> redv;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int C = d.C, V = d.V;
  const int r = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const RowStat* st = a.stats + static_cast<int64_t>(r) * C;
  const float T = temperature_of(d, r);
  const bool greedy = T == 0.f;  // row statistics were taken with s = 1: chunk maxima are the raw maxima
  const bool t_ok = greedy || temperature_ok(T);
  const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
  if (tid < 64) {
    float M;
    double D;
    combine_row(st, C, &M, &D);
    const RowNorm nn = make_norm(M, D);
    const bool ok = t_ok && norm_ok(nn);
    int cstar = -1;
    double tin = 0.0;
    if (ok && greedy) {
      for (int c0 = 0; c0 < C && cstar < 0; c0 += 64) {
        const int cc = c0 + lane;
        const uint64_t hit = __ballot(cc < C && st[cc].m == M);
        if (hit) cstar = c0 + __ffsll(static_cast<long long>(hit)) - 1;
      }
    } else if (ok) {
      const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(r), 0ull, a.offset, 1ull, a.seed, 0ull);
      cstar = select_chunk(C, u24(g.w[0]), [&](int cc) -> double { return stat_mass(st, cc, nn); }, &tin);
    }
    if (lane == 0) {
      sh.nrm = nn;
      sh.ok = ok ? 1 : 0;
      sh.cstar = cstar;
      sh.tin = tin;
    }
  }
  __syncthreads();
  int bb;
  bool al;
  const raw* row = row_of<E>(d, r, &bb, &al);
  int token = -1;
  if (sh.ok && sh.cstar >= 0) {
    if (greedy) {
      const int v = first_index_of<E, NT, S>(row, al, sh.cstar, sh.nrm.M, V, d.ntiles, red1);
      token = v == 0x7fffffff ? -1 : v;
    } else {
      token = sample_in_chunk<E, NT, S>(row, al, row, al, false, -1, sh.cstar, sh.tin, V, d.ntiles, s, sh.nrm,
                                        sh.nrm, kNoResidual, redv, red1, sh.smp);
    }
  }
  if (tid == 0) {
    a.token[r] = token;
    if (a.logz)
      a.logz[r] = (sh.ok && !greedy)
                      ? static_cast<float>((static_cast<double>(sh.nrm.M) + log2(sh.nrm.D)) * kLn2D)
                      : NAN;
  }
}

// ---------------------------------------------------------------------------
// per-step diagnostics

// One sub-chunk of one row.  With a_v = z_v s (log2 units) and the reference m:
// D = sum 2^(a_v - m), Em = sum 2^(a_v - m) (a_v - m), so that over a whole
// row with reference M the entropy in nats is ln2 (log2 D - Em / D).
struct DiagStat {
  float m;     // largest lane reference (log2 units), -inf: sub-chunk without mass
  float zmax;  // largest logit of the sub-chunk
  int arg;     // its first index
  int pad;
  double D;
  double Em;
};

struct DiagRow {   // one row, combined
  double H;        // entropy in nats
  float zmax;
  int arg;
};

struct DiagPair {  // one sub-chunk of a (target, draft) pair
  double gt;       // sum over p > q of q
  double ge;       // sum over q >= p of p
};

constexpr int kDiagCols = 7;  // column order of the per-step output

struct DiagArgs {
  RowsDesc rows;   // target rows (b, i < K) with tper = K, then draft rows, dper = K
  int B, K;
  float* out;      // [B, K, kDiagCols]
  int32_t* greedy; // [B, K] or null
  int32_t* prefer; // [B, K] or null
  const DiagStat* stats;  // [2BK][C]
  RowNorm* norms;         // [2BK]
  DiagRow* info;          // [2BK]
  DiagPair* pairs;        // [BK][C]
};

// Per-sub-chunk diagnostics statistics, one wave per sub-chunk: sub-chunk
// g = blockIdx.x * kWaves + wave of the rows' C sub-chunks each (row g / C,
// sub-chunk g % C) covers ST tiles of 256 vectors, i.e. ST * 4 vectors of the
// wave's 64 lanes, streamed S vectors per lane at a time.  Per lane: a running
// reference r (the largest z * s so far), D = sum 2^(z s - r) and the entropy
// moment E = sum 2^(z s - r) (z s - r), both rescaled when r grows, and the
// largest logit with the load step where it first appears.  Then one wave
// maximum of r and of the largest logit, float64 wave sums of the rescaled D
// and E, and the first index of the largest logit from the lanes that hold it
// (each reads that one load step again, from cache): no LDS, no barrier.
template <class E, int ST, int S>
__global__ __launch_bounds__(kThreads) void diag_stats_wave_kernel(RowsDesc d, DiagStat* __restrict__ stats,
                                                                   int64_t nsub) {
  constexpr int EPV = E::EPV;
  constexpr int WV = ST * (kThreads / 64);
  static_assert(WV % S == 0, "whole load steps per sub-chunk");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kWaves + wave;
  if (g >= nsub) return;  // the whole wave leaves: nothing below synchronises the workgroup
  const int C = d.C;
  const int r = static_cast<int>(g / C), j = static_cast<int>(g - static_cast<int64_t>(g / C) * C);
  int b;
  bool aligned;
  const typename E::raw* row = row_of<E>(d, r, &b, &aligned);
  const float T = temperature_of(d, b);
  const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
  const int e0 = j * WV * 64 * EPV;
  float ref = -INFINITY, dsum = 0.f, esum = 0.f, zmax = -INFINITY;
  int zstep = -1;
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
    if (mx > zmax) { zmax = mx; zstep = st; }
    const float nr = fmaxf(ref, mx * s);
    if (nr != -INFINITY) {
      float acc = 0.f, acce = 0.f;
#pragma unroll
      for (int i = 0; i < S; ++i)
#pragma unroll
        for (int k = 0; k < EPV; ++k) {
          const float tv = fmaf(x[i][k], s, -nr);
          const float e = __builtin_amdgcn_exp2f(tv);
          acc += e;
          // e * tv, with a masked token's -inf exponent clamped so that 0 * tv stays 0
          acce = fmaf(e, fmaxf(tv, -FLT_MAX), acce);
        }
      if (ref == -INFINITY) {
        dsum = acc; esum = acce;
      } else {  // nr >= ref: bring the running sums to the new reference
        const float sh = ref - nr;
        const float f = __builtin_amdgcn_exp2f(sh);
        esum = f * (esum + sh * dsum) + acce;
        dsum = dsum * f + acc;
      }
      ref = nr;
    }
  }
  const float m = wave_max(ref);
  const float zm = wave_max(zmax);
  double dd = 0.0, de = 0.0;
  if (dsum != dsum || esum != esum) {
    dd = NAN;  // data error propagates
  } else if (ref != -INFINITY) {
    const double f = static_cast<double>(__builtin_amdgcn_exp2f(ref - m));
    const double sh = static_cast<double>(ref) - static_cast<double>(m);
    dd = static_cast<double>(dsum) * f;
    de = f * (static_cast<double>(esum) + sh * static_cast<double>(dsum));
  }
  dd = wave_sum(dd);
  de = wave_sum(de);
  // first index of the sub-chunk's largest logit: the lanes that hold it scan
  // the load step where it first appears, ascending
  int arg = 0x7fffffff;
  if (zmax == zm && zm != -INFINITY) {
#pragma unroll
    for (int st = 0; st < WV / S; ++st)
      if (st == zstep) {
        const int es = e0 + st * S * 64 * EPV;
        float x[S][EPV];
        load_span<E, S, 64>(row, es, lane, d.V, aligned, x);
#pragma unroll
        for (int i = S - 1; i >= 0; --i)
#pragma unroll
          for (int k = EPV - 1; k >= 0; --k)
            if (x[i][k] == zm) arg = es + i * 64 * EPV + lane * EPV + k;
      }
  }
  arg = wave_min_int(arg);
  if (lane == 0) {
    DiagStat o;
    o.m = m; o.zmax = zm; o.arg = arg; o.pad = 0; o.D = dd; o.Em = de;
    stats[g] = o;
  }
}

// Split overlap sums, one wave per (pair, sub-chunk) item: item g = u * C + j
// is sub-chunk j of pair u (target row u, draft row B*K + u of the
// diagnostics row layout); gt = sum over p > q of q, ge = sum over q >= p of
// p, S vectors of each row per lane per load step, then float64 wave sums.
// One exponential per element pair: with x = log2 p and y = log2 q,
// 2^min(x, y) is q where x > y and p elsewhere, so x > y routes it.
template <class E, int ST, int S>
__global__ __launch_bounds__(kThreads) void diag_pair_wave_kernel(DiagArgs a, int64_t nitems) {
  constexpr int EPV = E::EPV;
  constexpr int WV = ST * (kThreads / 64);
  static_assert(WV % S == 0, "whole load steps per sub-chunk");
  const RowsDesc& d = a.rows;
  const int C = d.C, BK = a.B * a.K;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kWaves + wave;
  if (g >= nitems) return;  // the whole wave leaves: nothing below synchronises the workgroup
  const int u = static_cast<int>(g / C), j = static_cast<int>(g - static_cast<int64_t>(g / C) * C);
  int b;
  bool al_t, al_d;
  const typename E::raw* rt = row_of<E>(d, u, &b, &al_t);
  const typename E::raw* rd = row_of<E>(d, BK + u, &b, &al_d);
  const float T = temperature_of(d, b);
  const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
  const RowNorm nt = a.norms[u], nd = a.norms[BK + u];
  const int e0 = j * WV * 64 * EPV;
  float gt = 0.f, ge = 0.f;
#pragma unroll
  for (int st = 0; st < WV / S; ++st) {
    const int es = e0 + st * S * 64 * EPV;
    if (es >= d.V) break;  // wave-uniform: the row's last sub-chunk may be short
    float xt[S][EPV], xd[S][EPV];
    load_span<E, S, 64>(rt, es, lane, d.V, al_t, xt);
    load_span<E, S, 64>(rd, es, lane, d.V, al_d, xd);
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        const float lp = fmaf(xt[i][k], s, -nt.M) - nt.L;
        const float lq = fmaf(xd[i][k], s, -nd.M) - nd.L;
        const float mn = __builtin_amdgcn_exp2f(fminf(lp, lq));
        if (lp > lq) gt += mn;
        else ge += mn;
      }
  }
  const double vgt = wave_sum(static_cast<double>(gt));
  const double vge = wave_sum(static_cast<double>(ge));
  if (lane == 0) {
    DiagPair o;
    o.gt = vgt; o.ge = vge;
    a.pairs[g] = o;
  }
}

// One wave per row: normaliser, entropy, largest logit and its first index.
__global__ __launch_bounds__(kThreads) void diag_norm_kernel(const DiagStat* __restrict__ stats, int rows, int C,
                                                             RowNorm* __restrict__ norms, DiagRow* __restrict__ info) {
  const int r = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int lane = threadIdx.x & 63;
  const DiagStat* st = stats + static_cast<int64_t>(r) * C;
  float m = -INFINITY, zm = -INFINITY;
  for (int cc = lane; cc < C; cc += 64) {
    m = fmaxf(m, st[cc].m);
    zm = fmaxf(zm, st[cc].zmax);
  }
  m = wave_max(m);
  zm = wave_max(zm);
  double D = 0.0, Em = 0.0;
  int arg = 0x7fffffff;
  for (int cc = lane; cc < C; cc += 64) {
    const DiagStat sc = st[cc];
    if (sc.D != sc.D) {
      D += sc.D;
    } else if (sc.m != -INFINITY) {
      const double f = static_cast<double>(__builtin_amdgcn_exp2f(sc.m - m));
      D += sc.D * f;
      Em += f * (sc.Em + (static_cast<double>(sc.m) - static_cast<double>(m)) * sc.D);
    }
    if (sc.zmax == zm) arg = min(arg, sc.arg);
  }
  D = wave_sum(D);
  Em = wave_sum(Em);
  arg = wave_min_int(arg);
  if (lane == 0) {
    norms[r] = make_norm(m, D);
    DiagRow o;
    o.H = (log2(D) - Em / D) * kLn2D;
    o.zmax = zm;
    o.arg = arg;
    info[r] = o;
  }
}

// One wave per (b, i): every output of the step.
template <class E>
__global__ __launch_bounds__(kThreads) void diag_finish_kernel(DiagArgs a) {
  using raw = typename E::raw;
  const RowsDesc& d = a.rows;
  const int C = d.C, BK = a.B * a.K;
  const int u = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (u >= BK) return;
  const int lane = threadIdx.x & 63;
  const DiagPair* ps = a.pairs + static_cast<int64_t>(u) * C;
  double gt = 0.0, ge = 0.0;
  for (int cc = lane; cc < C; cc += 64) {
    gt += ps[cc].gt;
    ge += ps[cc].ge;
  }
  gt = wave_sum(gt);
  ge = wave_sum(ge);
  if (lane != 0) return;
  int b;
  bool al;
  const raw* rt = row_of<E>(d, u, &b, &al);
  const float T = temperature_of(d, b);
  const RowNorm nt = a.norms[u], nd = a.norms[BK + u];
  const DiagRow it = a.info[u], id = a.info[BK + u];
  const bool ok = temperature_ok(T) && norm_ok(nt) && norm_ok(nd);
  float* o = a.out + static_cast<int64_t>(u) * kDiagCols;
  if (!ok) {
    for (int k = 0; k < kDiagCols; ++k) o[k] = NAN;
    if (a.greedy) a.greedy[u] = -1;
    if (a.prefer) a.prefer[u] = -1;
    return;
  }
  const double s = static_cast<double>(scale_of(T));
  const double max_p = exp2(static_cast<double>(it.zmax) * s - static_cast<double>(nt.M)) / nt.D;
  const double a_to = exp2(static_cast<double>(E::one(rt + id.arg)) * s - static_cast<double>(nt.M)) / nt.D;
  const double a_rs = gt + ge;
  o[0] = static_cast<float>(it.H);
  o[1] = static_cast<float>(id.H);
  o[2] = static_cast<float>(max_p);
  o[3] = static_cast<float>(a_to);
  o[4] = static_cast<float>(a_rs);
  o[5] = static_cast<float>(gt);
  o[6] = static_cast<float>(ge);
  if (a.greedy) a.greedy[u] = id.arg;
  if (a.prefer) a.prefer[u] = a_rs > a_to ? 1 : 0;
}

}  // namespace sv

// verify_kernel.h — chain rejection-sampling verification (paper Sec. 2.2,
// Eq. reject_sample; App. G.1, Alg. rs_multinomial) in four launches that
// never wait on each other inside a launch:
//
//   1 row_stats   (sv_device.h) every target and draft row, one wave per
//                 sub-chunk: per-sub-chunk (max reference, exp2 sum).
//   2 decide      one workgroup per batch row: each row's normaliser from its
//                 chunk statistics; the K accept tests in parallel lanes
//                 (float64, u q(x) < p(x) with the two gathered logits and
//                 Philox uniforms); accept length; every output except the
//                 overlaps and the resampled token.
//   3 pair_pass   every (target row i, draft row i) pair, one wave (or, for
//                 small launches of residual steps, one workgroup) per
//                 sub-chunk: overlap sum min(p, q); for the row's first
//                 rejected step also the residual sums (residual mass,
//                 sum (p - q), sum over p > q of q).  Bonus rows are not read
//                 again, and without an overlap output only each row's
//                 residual step is.
//   4 finish      one workgroup per batch row: overlaps; the normalisation
//                 correction of the residual; the sub-chunk whose cumulative
//                 residual (or bonus) mass crosses u' Z, found from the
//                 per-sub-chunk masses; only that one is read again to
//                 invert the CDF inside it (tile sums, thread scan, element
//                 scan).
#pragma once

#include "sv_device.h"

namespace sv {

struct PairStat {  // one sub-chunk of a (target, draft) pair
  double alpha;    // sum min(p, q)
  // the row's first rejected step only: with p, q from the row normalisers,
  double Z;        // sum max(0, p - q)
  double Sd;       // sum (p - q)
  double Qg;       // sum of q over the elements with p > q
};

// The residual max(0, p - q) of the first rejected step, per element, to
// float32 precision of the residual itself, also where p and q nearly agree
// (the paper's operating regime: acceptance 0.75-0.99, residual masses down
// to 1e-3).  d = log2 p - log2 q is formed from the exact logit difference,
// d = (z_t - z_d) s - c, with c = log2 Z_t - log2 Z_d the difference of the
// row normalisers in float64 (split into float32 hi + lo); then
// p - q = sign(d) max(p, q) (1 - 2^-|d|).  The row normalisers come from
// float32 element sums, so the two rows' normalisations are exact only to
// about 1e-7: scaling p by rho = sum q / sum p (the sums of the same element
// values over the whole row) makes both sum to the same total, and the
// residual becomes max(0, (p - q) - p (1 - rho)).  1 - rho is itself formed
// from accurate sums, Sd / (alpha + Z) over the row's PairStat totals.
struct ResidualRef {
  float ch, cl;  // c = ch + cl
  float w;       // 1 - rho (0 while the pair pass forms the sums)
};

__device__ __forceinline__ ResidualRef residual_ref(const RowNorm& t, const RowNorm& d, double w) {
  const double c = (static_cast<double>(t.M) - static_cast<double>(d.M)) +
                   ((static_cast<double>(t.L) - static_cast<double>(d.L)) +
                    (static_cast<double>(t.Llo) - static_cast<double>(d.Llo)));
  ResidualRef r;
  r.ch = static_cast<float>(c);
  r.cl = static_cast<float>(c - static_cast<double>(r.ch));
  r.w = static_cast<float>(w);
  return r;
}

// The reference of a mass computation that is not a residual (p itself).
constexpr ResidualRef kNoResidual = {0.f, 0.f, 0.f};

// Signed p - q of one element and its min(p, q) and max(p, q), from the
// logits: lp, lq the float32 log2 probabilities, d the accurate log ratio.
// Below |d| = 1/2, |p - q| = max(p, q) (1 - 2^-|d|) with the series of
// 1 - e^-y (y = |d| ln 2 < 0.35, terms to y^7: truncation below 6e-8 of the
// value); above it the difference of the two exponentials, whose ratio is
// then at most 2^-1/2, so their rounding is at most six times the exponentials'
// own relative error.
struct ElemPQ {
  float g;    // |p - q|
  float dd;   // the accurate log2 p - log2 q (its sign is the sign of p - q)
  float mn;   // min(p, q)
  float mx;   // max(p, q)
  bool pos;   // p > q by the accurate log ratio
  __device__ __forceinline__ float diff() const { return copysignf(g, dd); }  // p - q
};
__device__ __forceinline__ ElemPQ elem_pq(float zt, float zd, float s, const RowNorm& t, const RowNorm& d,
                                          const ResidualRef& rr) {
  const float lp = fmaf(zt, s, -t.M) - t.L;
  const float lq = fmaf(zd, s, -d.M) - d.L;
  ElemPQ e;
  e.dd = fmaf(zt - zd, s, -rr.ch) - rr.cl;
  e.pos = e.dd > 0.f;
  e.mx = __builtin_amdgcn_exp2f(fmaxf(lp, lq));
  const float mn = __builtin_amdgcn_exp2f(fminf(lp, lq));
  const float y = fabsf(e.dd) * 0.69314718f;
  float p = 1.f / 5040.f;
  p = fmaf(p, -y, 1.f / 720.f);
  p = fmaf(p, -y, 1.f / 120.f);
  p = fmaf(p, -y, 1.f / 24.f);
  p = fmaf(p, -y, 1.f / 6.f);
  p = fmaf(p, -y, 0.5f);
  p = fmaf(p, -y, 1.f);
  const bool small = y < 0.34657359f;  // |d| < 1/2
  // (both logits -inf: mx = mn = 0 and g = 0; one of them -inf: |d| = inf and
  // g = mx, the other probability)
  e.g = small ? e.mx * (y * p) : e.mx - mn;
  e.mn = small ? e.mx - e.g : mn;
  return e;
}

// The residual mass of one element with the normalisation correction.
__device__ __forceinline__ float residual_mass(float zt, float zd, float s, const RowNorm& t, const RowNorm& d,
                                               const ResidualRef& rr) {
  const ElemPQ e = elem_pq(zt, zd, s, t, d, rr);
  return e.pos ? fmaxf(e.g - e.mx * rr.w, 0.f) : 0.f;
}

struct VerifyArgs {
  RowsDesc rows;   // target rows: tper = K+1; draft rows: dper = K
  int B, K;
  const int32_t* ids;
  uint64_t seed, offset;
  int32_t* accept_len; int32_t* emitted;
  float* overlap; float* p_at; float* q_at; float* logz_t; float* logz_d;
  const RowStat* stats;   // [rows][C]
  RowNorm* norms;         // [rows]
  int32_t* decision;      // [B]: accept length n, or -1 for a row with a data error
  PairStat* pairs;        // [B*K][C]
  int want_z;             // pair_pass also sums the residual mass of the first rejected step
};

__device__ __forceinline__ int target_row(const VerifyArgs& a, int b, int i) { return b * (a.K + 1) + i; }
__device__ __forceinline__ int draft_row(const VerifyArgs& a, int b, int i) {
  return a.B * (a.K + 1) + b * a.K + i;
}

struct DecideShared {
  RowNorm nrm[2 * SPEC_MAX_K_DEV + 1];  // target rows 0..K, then draft rows 0..K-1
};

// The draft token of step i, its target and draft logits and the accept
// uniform u_i, held by lane i: requested and drawn before the normalisers are
// known (the loads and the Philox rounds overlap the combine).
struct DraftGather {
  int x;
  float zt, zd;
  double u;
};

template <class E>
__device__ __forceinline__ DraftGather gather_draft(const VerifyArgs& a, int b, int i) {
  const RowsDesc& d = a.rows;
  DraftGather g;
  g.x = a.ids[static_cast<int64_t>(b) * a.K + i];
  g.zt = 0.f;
  g.zd = 0.f;
  const Philox4x64 ph = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(i), a.offset, 0ull, a.seed, 0ull);
  g.u = u24(ph.w[0]);
  if (g.x >= 0 && g.x < d.V) {
    int bb;
    bool al;
    g.zt = E::one(row_of<E>(d, target_row(a, b, i), &bb, &al) + g.x);
    g.zd = E::one(row_of<E>(d, draft_row(a, b, i), &bb, &al) + g.x);
  }
  return g;
}

// Accept tests and every per-row output except the overlaps and emitted[n],
// for batch row b whose 2K+1 row normalisers are in sh.nrm, by one wave: lane
// i < K tests step i (float64, u q(x) < p(x), no division), two ballots give
// the row's error flag and its first rejection, lane j <= K writes the
// outputs of position j (only with `write`: several workgroups may take the
// same decision, one of them writes it).  Returns the accept length n, or -1
// for a row with a data error (then every output of the row has been written).
// (T: the row's temperature.)
template <class E>
__device__ int decide_wave(const VerifyArgs& a, int b, const DecideShared& sh, const DraftGather& gx, float T,
                           bool write = true) {
  const RowsDesc& d = a.rows;
  const int K = a.K, V = d.V;
  const int lane = threadIdx.x & 63;
  const bool t_ok = temperature_ok(T);
  const float s = t_ok ? scale_of(T) : 1.0f;
  double p = 0.0, q = 0.0;
  bool ok = false, bad = false;
  if (lane < K) {
    const RowNorm& nt = sh.nrm[lane];
    const RowNorm& nd = sh.nrm[K + 1 + lane];
    bad = !(gx.x >= 0 && gx.x < V);
    if (!bad && t_ok && norm_ok(nt) && norm_ok(nd)) {
      p = exp2(static_cast<double>(gx.zt) * static_cast<double>(s) - static_cast<double>(nt.M)) / nt.D;
      q = exp2(static_cast<double>(gx.zd) * static_cast<double>(s) - static_cast<double>(nd.M)) / nd.D;
      ok = gx.u * q < p;
    }
  }
  const uint64_t errm = __ballot((lane < 2 * K + 1 && !norm_ok(sh.nrm[lane])) || bad);
  const uint64_t rejm = __ballot(lane < K && !ok);
  const bool err = !t_ok || errm != 0;
  // the first rejection ends the chain
  const int n = err ? -1 : (rejm ? __ffsll(static_cast<long long>(rejm)) - 1 : K);
  if (!write) return n;
  if (lane == 0) a.accept_len[b] = n;
  // the per-position outputs, one lane each (the float64 log2 of the normalisers in parallel)
  if (lane <= K) {
    const int j = lane;
    const int64_t ob = static_cast<int64_t>(b) * (K + 1) + j;
    // emitted[n] is written with the sampled token
    if (err || j != n) a.emitted[ob] = (!err && j < n) ? gx.x : -1;
    if (a.logz_t)
      a.logz_t[ob] = err ? NAN : static_cast<float>((static_cast<double>(sh.nrm[j].M) + log2(sh.nrm[j].D)) * kLn2D);
    if (j < K) {
      const int64_t o = static_cast<int64_t>(b) * K + j;
      const RowNorm& nd = sh.nrm[K + 1 + j];
      if (a.p_at) a.p_at[o] = err ? NAN : static_cast<float>(p);
      if (a.q_at) a.q_at[o] = err ? NAN : static_cast<float>(q);
      if (a.logz_d) a.logz_d[o] = err ? NAN : static_cast<float>((static_cast<double>(nd.M) + log2(nd.D)) * kLn2D);
      if (a.overlap && err) a.overlap[o] = NAN;
    }
  }
  return n;
}

// Row normalisers and accept decisions, one workgroup per batch row: every
// wave combines statistics of its rows, then wave 0 alone decides.
template <class E>
__global__ __launch_bounds__(kThreads) void decide_kernel(VerifyArgs a) {
  __shared__ DecideShared sh;
  const RowsDesc& d = a.rows;
  const int K = a.K, C = d.C;
  const int b = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  DraftGather gx{0, 0.f, 0.f, 0.0};
  if (static_cast<int>(threadIdx.x) < K) gx = gather_draft<E>(a, b, threadIdx.x);
  // row j < K+1: target row j; row K+1+i: draft row i (one wave per row, the
  // rows of a wave combined together so that their loads are in flight at once)
  const int R = 2 * K + 1;
  for (int j = wave; j < R; j += 2 * kWaves) {
    const int j2 = j + kWaves;
    const int r1 = j <= K ? target_row(a, b, j) : draft_row(a, b, j - K - 1);
    const int r2 = j2 < R ? (j2 <= K ? target_row(a, b, j2) : draft_row(a, b, j2 - K - 1)) : r1;
    float M1, M2;
    double D1, D2;
    combine_two_rows(a.stats + static_cast<int64_t>(r1) * C, a.stats + static_cast<int64_t>(r2) * C, C, &M1, &D1,
                     &M2, &D2);
    if (lane == 0) {
      const RowNorm n1 = make_norm(M1, D1);
      sh.nrm[j] = n1;
      a.norms[r1] = n1;
      if (j2 < R) {
        const RowNorm n2 = make_norm(M2, D2);
        sh.nrm[j2] = n2;
        a.norms[r2] = n2;
      }
    }
  }
  __syncthreads();
  if (wave != 0) return;  // the decision is one wave's work
  const int n = decide_wave<E>(a, b, sh, gx, temperature_of(d, b));
  if (lane == 0) a.decision[b] = n;
}

// Overlaps over one chunk of a (target, draft) pair, one workgroup per chunk
// (Gumbel-max verification, whose token needs no residual mass).
template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void pair_pass_kernel(VerifyArgs a, int64_t ntasks) {
  constexpr int EPV = E::EPV;
  __shared__ RedLds<4> red;
  const RowsDesc& d = a.rows;
  const int C = d.C;
  // grid-stride over the (pair, chunk) tasks (launched one workgroup per task)
  for (int64_t t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const int u = static_cast<int>(t / C), c = static_cast<int>(t - static_cast<int64_t>(t / C) * C);
    const int b = u / a.K, i = u % a.K;
    const int n = a.decision[b];
    if (n < 0) continue;  // data error: the finish ignores this row's partials
    const int rt_i = target_row(a, b, i), rd_i = draft_row(a, b, i);
    int bb;
    bool al_t, al_d;
    const typename E::raw* rt = row_of<E>(d, rt_i, &bb, &al_t);
    const typename E::raw* rd = row_of<E>(d, rd_i, &bb, &al_d);
    const float s = scale_of(temperature_of(d, b));
    const RowNorm nt = a.norms[rt_i], nd = a.norms[rd_i];
    const int tile0 = c * NT;
    const int nt_tiles = min(NT, d.ntiles - tile0);
    float al = 0.f;
#pragma unroll
    for (int j0 = 0; j0 < NT; j0 += S) {
      if (j0 >= nt_tiles) break;
      float xt[S][EPV], xd[S][EPV];
      load_tiles<E, S>(rt, tile0 + j0, d.V, al_t, xt);
      load_tiles<E, S>(rd, tile0 + j0, d.V, al_d, xd);
#pragma unroll
      for (int j = 0; j < S; ++j)
#pragma unroll
        for (int k = 0; k < EPV; ++k) al += min_prob(xt[j][k], xd[j][k], s, nt, nd);
    }
    double v[4] = {static_cast<double>(al), 0.0, 0.0, 0.0};
    wg_sum<4>(v, red);
    if (threadIdx.x == 0) {
      PairStat o;
      o.alpha = v[0]; o.Z = 0.0; o.Sd = 0.0; o.Qg = 0.0;
      a.pairs[t] = o;
    }
  }
}

// The pair-pass sums of one lane over one load step (S vectors of each row
// at element es): the overlap, and for the residual step the residual sums,
// in float32.
struct StepSums {
  float v[4];  // overlap, residual mass, sum of p - q, sum over p > q of q
};

template <class E, int S>
__device__ __forceinline__ StepSums pair_step_sums(const typename E::raw* rt, const typename E::raw* rd, bool al_t,
                                                   bool al_d, int es, int lane, int V, float s, const RowNorm& nt,
                                                   const RowNorm& nd, bool need_z, const ResidualRef& rr, float rft,
                                                   float rfd) {
  constexpr int EPV = E::EPV;
  StepSums o = {{0.f, 0.f, 0.f, 0.f}};
  float xt[S][EPV], xd[S][EPV];
  load_span<E, S, 64>(rt, es, lane, V, al_t, xt);
  load_span<E, S, 64>(rd, es, lane, V, al_d, xd);
  if (need_z) {
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        const ElemPQ e = elem_pq(xt[q][k], xd[q][k], s, nt, nd, rr);
        o.v[0] += e.mn;
        o.v[1] += e.pos ? e.g : 0.f;
        o.v[2] += e.diff();
        o.v[3] += e.pos ? e.mn : 0.f;
      }
  } else {
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int k = 0; k < EPV; ++k) o.v[0] += overlap_term<E>(xt[q][k], xd[q][k], s, nt, nd, rft, rfd);
  }
  return o;
}

// Pass 2 over (pair, sub-chunk) items.  Sub-chunk j covers ST tiles of 256
// vectors (ST * 4 vectors per lane of one wave), read in NS load steps of S
// vectors per lane.  Every item's sums are formed the same way, whichever
// launch shape runs it: per lane and load step in float32, per lane over the
// load steps in float64 (in step order), then one float64 sum over the
// wave's lanes.
//
// Two item orders.  Longest first (longest_first != 0): items 0 .. B*C-1
// are the sub-chunks of each batch row's residual step (its first rejected
// step, or step K-1 of a row that accepts every draft), the B*(K-1)*C items
// after them the rows' other steps (item (b*(K-1) + m)*C + j is sub-chunk j
// of the m-th of row b's other steps): a residual item costs about three
// times an overlap item, and taking them first keeps them from piling up at
// the end of a launch the device holds at once.  Pair order (item
// (b*K + i)*C + j), for launches many times what the device holds: there the
// longest-first order would run a phase of residual items alone, bound by
// the VALU, before a phase bound by memory, while the pair order mixes them.
// Two launch shapes:
//  - split == 0: one wave per item, kWaves items per workgroup;
//  - split == 1 (small batches, where one wave per item leaves the device
//    with too few loads in flight and the residual items' serial latency
//    bounds the launch): one workgroup per item, its kWaves waves sharing
//    the item's load steps and handing their per-lane step sums to wave 0
//    through LDS.
// Without overlaps only the residual-step items are launched.
// (The kernel runs each of its waves' items through pair_item, as a
// wave-stride loop for split == 0; in this form the compiler schedules the
// item's loads so that the pass runs 3-4 us faster at the B=256 batch, same
// bits.)
template <class E, int ST, int S>
__device__ __forceinline__ void pair_item(const VerifyArgs& a, int64_t nitems, int split, int longest_first,
                                          int64_t g_wave);
template <class E, int ST, int S>
__global__ __launch_bounds__(kThreads) void pair_pass_wave_kernel(VerifyArgs a, int64_t nitems, int split,
                                                                  int longest_first) {
  if (split) {
    pair_item<E, ST, S>(a, nitems, split, longest_first, -1);
    return;
  }
  const int wave = threadIdx.x >> 6;
  for (int64_t g = static_cast<int64_t>(blockIdx.x) * kWaves + wave; g < nitems;
       g += static_cast<int64_t>(gridDim.x) * kWaves)
    pair_item<E, ST, S>(a, nitems, split, longest_first, g);
}

// One item (split == 0: item g_wave of this wave; split == 1: item blockIdx.x
// of the whole workgroup).
template <class E, int ST, int S>
__device__ __forceinline__ void pair_item(const VerifyArgs& a, int64_t nitems, int split, int longest_first,
                                          int64_t g_wave) {
  constexpr int EPV = E::EPV;
  constexpr int WV = ST * (kThreads / 64);
  constexpr int NS = WV / S;  // load steps per sub-chunk
  static_assert(WV % S == 0 && NS % kWaves == 0, "whole load steps per sub-chunk and wave");
  __shared__ float part[NS][4][64];
  const RowsDesc& d = a.rows;
  const int C = d.C;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t first = static_cast<int64_t>(a.B) * C;
  const bool shared_item = split != 0;
  const int64_t g = shared_item ? static_cast<int64_t>(blockIdx.x) : g_wave;
  if (g >= nitems) return;  // (uniform over a workgroup that shares its item)
  int b, i, j;
  bool need_z;
  if (longest_first) {
    int m = 0;
    if (g < first) {
      b = static_cast<int>(g / C);
      j = static_cast<int>(g - static_cast<int64_t>(b) * C);
    } else {
      const int64_t g2 = g - first, per = static_cast<int64_t>(a.K - 1) * C;
      b = static_cast<int>(g2 / per);
      const int r = static_cast<int>(g2 - static_cast<int64_t>(b) * per);
      m = r / C;
      j = r - m * C;
    }
    const int n = a.decision[b];
    if (n < 0) return;  // data error: finish ignores this row's partials
    const bool rejects = a.want_z && n < a.K;
    const int i0 = rejects ? n : a.K - 1;
    i = g < first ? i0 : (m < i0 ? m : m + 1);
    need_z = rejects && g < first;
  } else {  // pair order: item g = (b * K + i) * C + j
    const int u = static_cast<int>(g / C);
    j = static_cast<int>(g - static_cast<int64_t>(u) * C);
    b = u / a.K;
    i = u - b * a.K;
    const int n = a.decision[b];
    if (n < 0) return;
    need_z = a.want_z && i == n;
  }
  // (all of the above is uniform over a workgroup that shares its item, so
  // the returns leave its barrier to all of its waves or to none)
  if (!need_z && a.overlap == nullptr) return;  // no overlap requested: only the residual step is read again
  const int rt_i = target_row(a, b, i), rd_i = draft_row(a, b, i);
  int bb;
  bool al_t, al_d;
  const typename E::raw* rt = row_of<E>(d, rt_i, &bb, &al_t);
  const typename E::raw* rd = row_of<E>(d, rd_i, &bb, &al_d);
  const float s = scale_of(temperature_of(d, b));
  const RowNorm nt = a.norms[rt_i], nd = a.norms[rd_i];
  const ResidualRef rr = need_z ? residual_ref(nt, nd, 0.0) : kNoResidual;
  const float rft = static_cast<float>(static_cast<double>(nt.M) + static_cast<double>(nt.L));
  const float rfd = static_cast<float>(static_cast<double>(nd.M) + static_cast<double>(nd.L));
  const int e0 = j * WV * 64 * EPV;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  if (shared_item) {
    constexpr int NW = NS / kWaves;
#pragma unroll 1
    for (int st = wave * NW; st < (wave + 1) * NW; ++st) {
      const int es = e0 + st * S * 64 * EPV;
      StepSums ps = {{0.f, 0.f, 0.f, 0.f}};
      if (es < d.V) ps = pair_step_sums<E, S>(rt, rd, al_t, al_d, es, lane, d.V, s, nt, nd, need_z, rr, rft, rfd);
#pragma unroll
      for (int q = 0; q < 4; ++q) part[st][q][lane] = ps.v[q];
    }
    __syncthreads();
    if (wave != 0) return;
    // (a step beyond the row adds +0, as the one-wave shape skips it)
#pragma unroll
    for (int st = 0; st < NS; ++st)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[q] += static_cast<double>(part[st][q][lane]);
  } else if (need_z) {
    // (a loop that is not unrolled, so that its longer body does not
    // multiply the code size)
#pragma unroll 1
    for (int st = 0; st < NS; ++st) {
      const int es = e0 + st * S * 64 * EPV;
      if (es >= d.V) break;  // wave-uniform: the row's last sub-chunk may be short
      const StepSums ps = pair_step_sums<E, S>(rt, rd, al_t, al_d, es, lane, d.V, s, nt, nd, true, rr, rft, rfd);
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[q] += static_cast<double>(ps.v[q]);
    }
  } else {
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int es = e0 + st * S * 64 * EPV;
      if (es >= d.V) break;  // wave-uniform: the row's last sub-chunk may be short
      const StepSums ps = pair_step_sums<E, S>(rt, rd, al_t, al_d, es, lane, d.V, s, nt, nd, false, rr, rft, rfd);
      acc[0] += static_cast<double>(ps.v[0]);
    }
  }
  PairStat o;
  o.alpha = wave_sum(acc[0]);
  o.Z = need_z ? wave_sum(acc[1]) : 0.0;
  o.Sd = need_z ? wave_sum(acc[2]) : 0.0;
  o.Qg = need_z ? wave_sum(acc[3]) : 0.0;
  if (lane == 0) a.pairs[(static_cast<int64_t>(b) * a.K + i) * C + j] = o;
}

// Residual (or target) mass of the EPV elements of one thread's vector;
// element `excl` (-1: none) has mass 0.
template <class E>
__device__ __forceinline__ void vector_masses(const typename E::raw* rt, const typename E::raw* rd, bool residual,
                                              int excl, int v0, int V, float s, const RowNorm& nt,
                                              const RowNorm& nd, const ResidualRef& rr, float (&r)[E::EPV]) {
#pragma unroll
  for (int k = 0; k < E::EPV; ++k) {
    if (v0 + k < V && v0 + k != excl) {
      const float zt = E::one(rt + v0 + k);
      r[k] = residual ? residual_mass(zt, E::one(rd + v0 + k), s, nt, nd, rr) : prob(zt, s, nt.M, nt.invD);
    } else {
      r[k] = 0.f;
    }
  }
}

// The chunk holding the sampling target, found by one wave from per-chunk
// masses mass(cc) >= 0: with the total Z and the uniform u, target = u Z; the
// chunk is the first whose cumulative mass exceeds the target (strict ">", so
// a chunk without mass is never chosen).  *tin receives the target's offset
// inside the chunk; if rounding puts the target past the last cumulative sum,
// the last chunk with mass is chosen and *tin = +inf (its last element with
// mass).  Returns -1 when no chunk has mass.
template <class Mass>
__device__ __forceinline__ int select_chunk(int C, double u, Mass mass, double* tin) {
  const int lane = threadIdx.x & 63;
  double tot = 0.0;
  for (int cc = lane; cc < C; cc += 64) tot += mass(cc);
  tot = wave_sum(tot);
  const double target = u * tot;
  double carry = 0.0, t_in = 0.0;
  int cstar = -1, clast = -1;
  for (int c0 = 0; c0 < C; c0 += 64) {
    const int cc = c0 + lane;
    const double zc = (cc < C) ? mass(cc) : 0.0;
    const double incl = carry + wave_incl_scan(zc);
    const double excl = incl - zc;
    const uint64_t hit = __ballot(cc < C && incl > target && excl <= target && zc > 0.0);
    const uint64_t pos = __ballot(cc < C && zc > 0.0);
    if (pos) clast = c0 + 63 - __clzll(pos);
    if (cstar < 0 && hit) {
      const int l = __ffsll(static_cast<long long>(hit)) - 1;
      cstar = c0 + l;
      t_in = target - __shfl(excl, l, 64);
    }
    carry = __shfl(incl, 63, 64);
  }
  if (cstar < 0) { cstar = clast; t_in = INFINITY; }
  *tin = t_in;
  return cstar;
}

struct SampleShared {
  int token;
};

// Per-tile masses of chunk `c` (NT tiles of kThreads vectors, read S tiles at
// a time), per thread: tsum[j] = this thread's mass in tile j.  The mass of an
// element is the residual max(0, p - q) with the normalisation correction
// (`residual`, residual_mass), else p; element `excl` (-1: none) has mass 0.
// Returns the number of tiles in the chunk.
template <class E, int NT, int S>
__device__ __forceinline__ int tile_masses(const typename E::raw* rt, bool al_t, const typename E::raw* rd,
                                           bool al_d, bool residual, int excl, int c, int V, int ntiles, float s,
                                           const RowNorm& nt, const RowNorm& nd, const ResidualRef& rr,
                                           float (&tsum)[NT], float (*keep)[S][E::EPV] = nullptr) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  const int tile0 = c * NT;
  const int nt_tiles = min(NT, ntiles - tile0);
  // the excluded element, as (tile, lane of this thread's vector), or none
  const int ex_rel = excl - tile0 * TILE;
  const int ex_tile = (excl >= 0 && ex_rel >= 0 && ex_rel < NT * TILE) ? ex_rel / TILE : -1;
  const int ex_k = (ex_tile >= 0 && (ex_rel % TILE) / EPV == static_cast<int>(threadIdx.x)) ? ex_rel % EPV : -1;
#pragma unroll
  for (int j = 0; j < NT; ++j) tsum[j] = 0.f;
#pragma unroll
  for (int j0 = 0; j0 < NT; j0 += S) {
    if (j0 >= nt_tiles) break;
    float xt[S][EPV], xd[S][EPV];
    load_tiles<E, S>(rt, tile0 + j0, V, al_t, xt);
    if (residual) load_tiles<E, S>(rd, tile0 + j0, V, al_d, xd);
#pragma unroll
    for (int j = 0; j < S; ++j)
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        float m = residual ? residual_mass(xt[j][k], xd[j][k], s, nt, nd, rr) : prob(xt[j][k], s, nt.M, nt.invD);
        if (j0 + j == ex_tile && k == ex_k) m = 0.f;
        tsum[j0 + j] += m;
        if (keep) (*keep)[j][k] = m;
      }
  }
  return nt_tiles;
}

// Inverse CDF inside chunk `cstar`, whole workgroup: per-tile masses
// (tile_masses), the tile holding `tin`, a workgroup scan of the per-thread
// masses of that tile, then an element scan in the winning thread.  Every
// thread returns the token (-1 if the chunk has no mass).
template <class E, int NT, int S>
__device__ int sample_in_chunk(const typename E::raw* rt, bool al_t, const typename E::raw* rd, bool al_d,
                               bool residual, int excl, int cstar, double tin, int V, int ntiles, float s,
                               const RowNorm& nt, const RowNorm& nd, const ResidualRef& rr, RedLds<NT>& redv,
                               RedLds<1>& red1, SampleShared& sh) {
  constexpr int EPV = E::EPV;
  constexpr int TILE = kThreads * EPV;
  const int tid = threadIdx.x;
  const int tile0 = cstar * NT;
  float tsum[NT];
  // a chunk of one load step keeps its element masses for the final scan
  float keep[S][EPV];
  const int nt_tiles = tile_masses<E, NT, S>(rt, al_t, rd, al_d, residual, excl, cstar, V, ntiles, s, nt, nd, rr,
                                             tsum, NT == S ? &keep : nullptr);
  double W[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) W[j] = (j < nt_tiles) ? static_cast<double>(tsum[j]) : 0.0;
  wg_sum<NT>(W, redv);  // tile totals, identical in every thread
  int jstar = -1, jlast = -1;
  double cum = 0.0, t_in = 0.0;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    if (j < nt_tiles) {
      if (W[j] > 0.0) jlast = j;
      if (jstar < 0 && cum + W[j] > tin) { jstar = j; t_in = tin - cum; }
      cum += W[j];
    }
  }
  bool clamp = false;
  if (jstar < 0) { jstar = jlast; clamp = true; }
  if (jstar < 0) return -1;
  float w = 0.f;
#pragma unroll
  for (int j = 0; j < NT; ++j)
    if (j == jstar) w = tsum[j];
  // the wave holding the target from the wave totals (one exchange through
  // LDS), then a prefix scan inside that wave only; its winning lane scans its
  // elements and writes the token
  const int wave = tid >> 6, lane = tid & 63;
  const double wt = wave_sum(static_cast<double>(w));
  if (lane == 0) red1.d[wave][0] = wt;
  if (tid == 0) sh.token = -1;
  __syncthreads();
  int twave = -1, tlast = -1;
  double tbase = 0.0, base = 0.0;
#pragma unroll
  for (int w2 = 0; w2 < kWaves; ++w2) {
    const double tw = red1.d[w2][0];
    if (tw > 0.0) tlast = w2;
    if (!clamp && twave < 0 && tw > 0.0 && base + tw > t_in) { twave = w2; tbase = base; }
    base += tw;
  }
  if (twave < 0) { clamp = true; twave = tlast; }  // rounding: the last wave with mass
  if (wave == twave) {
    const double incl = tbase + wave_incl_scan(static_cast<double>(w));
    const double excl_sum = incl - static_cast<double>(w);
    const uint64_t hit = clamp ? 0ull : __ballot(incl > t_in && excl_sum <= t_in && w > 0.f);
    bool lclamp = clamp;
    int lstar;
    if (hit) {
      lstar = __ffsll(static_cast<long long>(hit)) - 1;
    } else {  // rounding inside the wave: its last lane with mass
      lclamp = true;
      const uint64_t pos = __ballot(w > 0.f);
      lstar = pos ? 63 - __clzll(pos) : -1;
    }
    if (lane == lstar) {
      const int v0 = (tile0 + jstar) * TILE + tid * EPV;
      float r[EPV];
      if constexpr (NT == S) {
#pragma unroll
        for (int j = 0; j < NT; ++j)
          if (j == jstar)
#pragma unroll
            for (int k = 0; k < EPV; ++k) r[k] = keep[j][k];
      } else {
        vector_masses<E>(rt, rd, residual, excl, v0, V, s, nt, nd, rr, r);
      }
      const double tl = t_in - excl_sum;
      float cumf = 0.f;
      int kstar = -1, klast = -1;
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        cumf += r[k];
        if (r[k] > 0.f) klast = k;
        if (kstar < 0 && !lclamp && r[k] > 0.f && static_cast<double>(cumf) > tl) kstar = k;
      }
      if (kstar < 0) kstar = klast;
      if (kstar >= 0) sh.token = v0 + kstar;
    }
  }
  __syncthreads();
  return sh.token;
}

struct FinishShared {
  double alpha[SPEC_MAX_K_DEV];
  RowNorm nrm[2 * SPEC_MAX_K_DEV + 1];  // target rows 0..K, then draft rows 0..K-1
  double tin, w;
  int cstar, residual;
  SampleShared smp;
};

// The residual mass of one sub-chunk at the rejected step, with the
// normalisation correction w = 1 - rho: the elements with p > q lose p w
// each, sum_{p > q} p = Qg + Z.
__device__ __forceinline__ double corrected_mass(double z, double qg, double w) {
  return fmax(z - (qg + z) * w, 0.0);
}

// One workgroup per batch row: overlaps and the resampled / bonus token.
// Everything the row can need except the chosen sub-chunk is requested before
// its accept length is known, in one round trip: the overlap partials, the
// residual sums of every step and the bonus row's statistics for the first
// 64 sub-chunks, and the normalisers of the 2K+1 rows; the uniform of every
// possible emitting step is drawn meanwhile, one lane per step.  Then only the
// chosen sub-chunk is read.
template <class E, int NT, int S>
__global__ __launch_bounds__(kThreads) void finish_kernel(VerifyArgs a) {
  using raw = typename E::raw;
  __shared__ FinishShared sh;
  __shared__ RedLds<NT> redv;
  __shared__ RedLds<1> red1;
  const RowsDesc& d = a.rows;
  const int K = a.K, C = d.C, V = d.V;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  if (tid < 2 * K + 1) sh.nrm[tid] = a.norms[tid <= K ? target_row(a, b, tid) : draft_row(a, b, tid - K - 1)];
  // overlap partials of every draft step (one wave per step, sub-chunk order fixed)
  double al = 0.0;
  if (a.overlap != nullptr && wave < K) {
    const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + wave) * C;
    for (int cc = lane; cc < C; cc += 64) al += ps[cc].alpha;
  }
  // wave 0, lane cc < 64: sub-chunk cc's residual sums of every step and the
  // bonus row's statistics; lane j <= K: target row j's normaliser and the
  // uniform u' of step j
  PairStat ppre[SPEC_MAX_K_DEV];
  RowStat spre;
  spre.m = -INFINITY; spre.pad = 0.f; spre.D = 0.0;
  float nM = 0.f;
  double nD = 1.0, uq = 0.0;
  if (wave == 0) {
#pragma unroll
    for (int i = 0; i < SPEC_MAX_K_DEV; ++i) {
      ppre[i].alpha = 0.0; ppre[i].Z = 0.0; ppre[i].Sd = 0.0; ppre[i].Qg = 0.0;
      if (i < K && lane < C) ppre[i] = a.pairs[static_cast<int64_t>(b * K + i) * C + lane];
    }
    if (lane < C) spre = a.stats[static_cast<int64_t>(target_row(a, b, K)) * C + lane];
    if (lane <= K) {
      const RowNorm nl = a.norms[target_row(a, b, lane)];
      nM = nl.M;
      nD = nl.D;
      const Philox4x64 g = philox4x64_10(static_cast<uint64_t>(b), static_cast<uint64_t>(lane), a.offset, 0ull,
                                         a.seed, 0ull);
      uq = u24(g.w[1]);
    }
  }
  const int n = a.decision[b];
  if (n < 0) return;  // data error: decide has written every output of the row
  const float s = scale_of(temperature_of(d, b));

  if (a.overlap != nullptr && wave < K) {
    al = wave_sum(al);
    if (lane == 0) sh.alpha[wave] = al;
    for (int i = wave + kWaves; i < K; i += kWaves) {  // K > kWaves: the remaining steps
      double al2 = 0.0;
      const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + i) * C;
      for (int cc = lane; cc < C; cc += 64) al2 += ps[cc].alpha;
      al2 = wave_sum(al2);
      if (lane == 0) sh.alpha[i] = al2;
    }
  }
  // the sub-chunk holding the sampling target (wave 0)
  if (wave == 0) {
    const PairStat* ps = a.pairs + static_cast<int64_t>(b * K + (n < K ? n : 0)) * C;
    PairStat p0;
    p0.alpha = 0.0; p0.Z = 0.0; p0.Sd = 0.0; p0.Qg = 0.0;
#pragma unroll
    for (int i = 0; i < SPEC_MAX_K_DEV; ++i)
      if (i == n) p0 = ppre[i];
    // the row's totals at the rejected step, and its normalisation correction
    double w = 0.0;
    bool any_residual = false;
    if (n < K) {
      double za = 0.0, zd = 0.0, zal = 0.0;
      for (int cc = lane; cc < C; cc += 64) {
        const PairStat q = cc < 64 ? p0 : ps[cc];
        za += q.Z; zd += q.Sd; zal += q.alpha;
      }
      za = wave_sum(za);
      zd = wave_sum(zd);
      zal = wave_sum(zal);
      w = zd / (zal + za);
      if (!(w == w)) w = 0.0;
      bool pos = false;
      for (int cc = lane; cc < C; cc += 64) {
        const PairStat q = cc < 64 ? p0 : ps[cc];
        pos = pos || corrected_mass(q.Z, q.Qg, w) > 0.0;
      }
      any_residual = __ballot(pos) != 0;
    }
    // residual of the rejected step; p_n itself for the bonus row or an empty residual
    const bool residual = n < K && any_residual;
    const RowStat* st = a.stats + static_cast<int64_t>(target_row(a, b, n)) * C;
    const float nnM = __shfl(nM, n, 64);
    const double nnD = __shfl(nD, n, 64);
    // this lane's mass of sub-chunk `lane` (select_chunk asks for cc = c0 + lane,
    // c0 a multiple of 64; beyond the first 64 sub-chunks they are read)
    auto stat_mass1 = [&](const RowStat& sc) -> double {
      return sc.m == -INFINITY ? 0.0 : sc.D * static_cast<double>(__builtin_amdgcn_exp2f(sc.m - nnM)) / nnD;
    };
    const double m0 =
        lane < C ? (residual ? corrected_mass(p0.Z, p0.Qg, w) : stat_mass1(n == K ? spre : st[lane])) : 0.0;
    double tin;
    const int cstar = select_chunk(C, __shfl(uq, n, 64), [&](int cc) -> double {
      if (cc < 64) return m0;
      return residual ? corrected_mass(ps[cc].Z, ps[cc].Qg, w) : stat_mass1(st[cc]);
    }, &tin);
    if (lane == 0) {
      sh.cstar = cstar;
      sh.tin = tin;
      sh.residual = residual ? 1 : 0;
      sh.w = w;
    }
  }
  __syncthreads();

  int token = -1;
  if (sh.cstar >= 0) {
    int bb;
    bool al_t, al_d;
    const raw* rt = row_of<E>(d, target_row(a, b, n), &bb, &al_t);
    const raw* rd = row_of<E>(d, draft_row(a, b, n < K ? n : 0), &bb, &al_d);
    const RowNorm nt = sh.nrm[n];
    const RowNorm nd = sh.nrm[K + 1 + (n < K ? n : 0)];
    const ResidualRef rr = residual_ref(nt, nd, sh.w);
    token = sample_in_chunk<E, NT, S>(rt, al_t, rd, al_d, sh.residual != 0, -1, sh.cstar, sh.tin, V, d.ntiles, s, nt,
                                      nd, rr, redv, red1, sh.smp);
  }

  // the overlaps and emitted[n] have this single writer
  if (tid == 0) {
    a.emitted[static_cast<int64_t>(b) * (K + 1) + n] = token;
    if (a.overlap)
      for (int i = 0; i < K; ++i) a.overlap[static_cast<int64_t>(b) * K + i] = static_cast<float>(sh.alpha[i]);
  }
}

}  // namespace sv

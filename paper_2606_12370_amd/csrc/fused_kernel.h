// fused_kernel.h — rejection-sampling verification (paper Sec. 2.2, Eq.
// reject_sample; App. G.1, Alg. rs_multinomial) with a single read of the
// logits.
//
// Every batch row is spread over a group of G co-resident workgroups, one per
// slice of the vocabulary (2 tiles: 512 16-byte vectors, 4096 bf16 or 2048
// fp32 elements), and a group takes its batch rows one after another
// (group k: rows k, k + NG, ...).  Each workgroup runs a three-stage
// pipeline over its group's rows, one step per row:
//   1 issue the loads of the next row's slice of all 2K+1 rows (two vectors
//     per thread and row, with the row's temperature and draft tokens) into
//     one of two register sets;
//   2 reduce the current row's slice of each row to (max reference, exp2
//     sum) and publish the records with agent-scope atomic stores, then park
//     the slice's K pair rows (and the draft-token inputs of the decisions)
//     in LDS;
//   3 for the row parked one step earlier: wait for the G records of each of
//     its rows (published by the other workgroups of the group, which run at
//     the same time), combine them into the row normalisers in the fixed
//     order every kernel of the library uses, take the accept decisions
//     (every workgroup the same ones; the first writes them), and sum from
//     LDS the overlap of every draft step and the residual sums of the
//     residual step over its slice.
// A step issues its loads in the order they are waited for (the first poll
// of stage 3's records, the draft logits of stage 2's row, then stage 1), so
// that no wait for an older load also waits for the next row's slice.
// The finish launch (verify_kernel.h) then forms the overlaps, picks the
// slice holding the resampled token and inverts the CDF inside it.
//
// The record array is set to all-ones bits before the launch; a record is
// complete once neither of its two 64-bit words is all ones (a normaliser sum
// that is NaN is stored as the canonical NaN).  The launch is cooperative, so
// every workgroup of a group is resident while the others wait for it; each
// wait is still bounded by a spin limit, after which the row's normalisers
// are NaN and the row is reported as a data error.
#pragma once

#include "verify_kernel.h"

namespace sv {

constexpr int kFusedNV = 2;  // vectors per thread per row and slice
constexpr uint64_t kRecordEmpty = ~0ull;

__device__ __forceinline__ uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A vector of -inf elements: the slice's vectors past the end of the row (the
// path runs only on rows whose length is a multiple of the vector, so a
// vector lies wholly inside or wholly past it).
template <class E>
__device__ __forceinline__ typename E::vec neg_inf_vector() {
  const uint32_t h = E::EPV == 8 ? 0xFF80FF80u : 0xFF800000u;
  typename E::vec w;
  w.x = h;
  w.y = h;
  w.z = h;
  w.w = h;
  return w;
}

__global__ __launch_bounds__(kThreads) void fill_ones_kernel(uint64_t* __restrict__ p, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads)
    p[i] = kRecordEmpty;
}

// The pair rows of the batch row in its overlap stage, parked in LDS while
// the next batch row's statistics run: 2K rows x kFusedNV vectors per thread.
template <class E, int K>
struct FusedShared {
  typename E::vec pbuf[2 * K][kFusedNV][kThreads];
  DraftGather pgx[K];
  float2 part[2 * K + 1][kThreads];
  DecideShared dec;  // the 2K+1 row normalisers of the batch row in its overlap stage
  double pr[kWaves][SPEC_MAX_K_DEV + 3];
  float pT;  // temperature of the parked batch row
  int n, pb, gave_up;
};

// One batch row's slice of all 2K+1 rows as raw vectors, with what its
// decision needs (the draft token, its two logits and the accept uniform,
// held by lane i of wave 0 for step i).
template <class E, int K>
struct FusedUnit {
  typename E::vec w[2 * K + 1][kFusedNV];
  DraftGather gx;
  float T;  // the batch row's temperature
  int id;   // lane i < K: draft token of step i (other lanes: step 0's)
  int b;    // batch row, or -1 when the stage is empty
};

// The exchange records of a batch row's 2K+1 rows that one wave reads (rows
// wave, wave + 4, ...; lane g < G: member g's record), as first polled.
template <int K>
struct FusedPoll {
  static constexpr int RW = (2 * K + 1 + kWaves - 1) / kWaves;
  uint64_t w0[RW], w1[RW];
};

template <class E, int K>
struct FusedCtx {
  const VerifyArgs& a;
  int G, g, e0, tid, wave, lane;
  unsigned spin_limit;
  FusedShared<E, K>* sh;
  float temp_scalar;  // the temperature of every row when there is no per-row array
};

template <class E, int K>
__device__ __forceinline__ const typename E::raw* fused_row(const VerifyArgs& a, int b, int r) {
  using raw = typename E::raw;
  const RowsDesc& d = a.rows;
  return r <= K ? static_cast<const raw*>(d.tgt) + static_cast<int64_t>(b) * d.tsb + static_cast<int64_t>(r) * d.tsk
                : static_cast<const raw*>(d.drf) + static_cast<int64_t>(b) * d.dsb +
                      static_cast<int64_t>(r - K - 1) * d.dsk;
}

template <class E, int K>
__device__ __forceinline__ int fused_row_index(const VerifyArgs& a, int b, int r) {
  return r <= K ? target_row(a, b, r) : draft_row(a, b, r - K - 1);
}

// Every stage issues the same loads on every path (an empty stage or a lane
// past the group loads from row 0 and ignores the result), so that the
// compiler's wait counts stay exact: a wait for an older load never drains
// the loads issued after it.

// Stage 1: issue the loads of batch row b's slice (no wait): the
// temperature and the draft tokens first, then the 2K+1 rows.
template <class E, int K>
__device__ __forceinline__ void fused_load(const FusedCtx<E, K>& c, int b, FusedUnit<E, K>& u) {
  using vec = typename E::vec;
  constexpr int EPV = E::EPV;
  const VerifyArgs& a = c.a;
  u.b = b;
  const int bl = b < 0 ? 0 : b;
  const int V = a.rows.V;
  // (the value is selected, not the address: the per-row array is global
  // memory, the scalar a kernel argument read once at the start)
  const float* tp = a.rows.temp ? a.rows.temp + bl : reinterpret_cast<const float*>(a.ids);
  const float tv = *tp;
  u.T = a.rows.temp ? tv : c.temp_scalar;
  u.id = a.ids[static_cast<int64_t>(bl) * a.K + (c.lane < K ? c.lane : 0)];
#pragma unroll
  for (int r = 0; r < 2 * K + 1; ++r) {
    const typename E::raw* rp = fused_row<E, K>(a, bl, r);
#pragma unroll
    for (int j = 0; j < kFusedNV; ++j) {
      const int v0 = c.e0 + (j * kThreads + c.tid) * EPV;
      u.w[r][j] = __builtin_nontemporal_load(reinterpret_cast<const vec*>(rp + ((v0 + EPV <= V) ? v0 : 0)));
    }
  }
}

// The draft token's two logits and the step's accept uniform (lane i < K:
// step i), from the token loaded one stage earlier (no wait for the logits).
template <class E, int K>
__device__ __forceinline__ void fused_gather(const FusedCtx<E, K>& c, FusedUnit<E, K>& u) {
  const VerifyArgs& a = c.a;
  const int bl = u.b < 0 ? 0 : u.b;
  const int i = c.lane < K ? c.lane : 0;
  const int x = u.id;
  const int xs = (x >= 0 && x < a.rows.V) ? x : 0;
  u.gx.x = x;
  u.gx.zt = E::one(fused_row<E, K>(a, bl, i) + xs);
  u.gx.zd = E::one(fused_row<E, K>(a, bl, K + 1 + i) + xs);
  u.gx.u = 0.0;
  if (c.tid < K) {
    const Philox4x64 ph =
        philox4x64_10(static_cast<uint64_t>(bl), static_cast<uint64_t>(i), a.offset, 0ull, a.seed, 0ull);
    u.gx.u = u24(ph.w[0]);
  }
}

// The first poll of the exchange records of batch row b (no wait).
template <class E, int K>
__device__ __forceinline__ void fused_poll(const FusedCtx<E, K>& c, int b, FusedPoll<K>& pl) {
  const int bl = b < 0 ? 0 : b;
#pragma unroll
  for (int i = 0; i < FusedPoll<K>::RW; ++i) {
    const int r = c.wave + kWaves * i;
    const int row = fused_row_index<E, K>(c.a, bl, r < 2 * K + 1 ? r : 0);
    const uint64_t* rec = reinterpret_cast<const uint64_t*>(c.a.stats + static_cast<int64_t>(row) * c.G) +
                          2 * (c.lane < c.G ? c.lane : 0);
    pl.w0[i] = ld_agent(rec);
    pl.w1[i] = ld_agent(rec + 1);
  }
}

// Stage 2: reduce every row of the slice to (max reference, exp2 sum) and
// publish one record per row.
template <class E, int K>
__device__ __forceinline__ void fused_stats(const FusedCtx<E, K>& c, FusedUnit<E, K>& u) {
  constexpr int EPV = E::EPV;
  constexpr int R = 2 * K + 1;
  const VerifyArgs& a = c.a;
  FusedShared<E, K>& sh = *c.sh;
  const int b = u.b;
  const int V = a.rows.V;
  const float T = u.T;
  const float s = temperature_ok(T) ? scale_of(T) : 1.0f;
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int j = 0; j < kFusedNV; ++j) {
      const int v0 = c.e0 + (j * kThreads + c.tid) * EPV;
      if (v0 >= V) u.w[r][j] = neg_inf_vector<E>();
    }
    float x[kFusedNV][EPV];
#pragma unroll
    for (int j = 0; j < kFusedNV; ++j) E::widen(u.w[r][j], x[j]);
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kFusedNV; ++j)
#pragma unroll
      for (int k = 0; k < EPV; ++k) mx = fmaxf(mx, x[j][k]);
    const float ref = mx * s;
    float acc = 0.f;
    if (ref != -INFINITY) {
#pragma unroll
      for (int j = 0; j < kFusedNV; ++j)
#pragma unroll
        for (int k = 0; k < EPV; ++k) acc += __builtin_amdgcn_exp2f(fmaf(x[j][k], s, -ref));
    }
    sh.part[r][c.tid] = make_float2(ref, acc);
    // one row at a time: interleaving the rows would hold every row's
    // widened values at once
    __builtin_amdgcn_sched_barrier(0);
  }
  __syncthreads();
  for (int r = c.wave; r < R; r += kWaves) {
    float rf[kThreads / 64], ac[kThreads / 64];
    float m = -INFINITY;
#pragma unroll
    for (int q = 0; q < kThreads / 64; ++q) {
      const float2 pq = sh.part[r][c.lane + 64 * q];
      rf[q] = pq.x;
      ac[q] = pq.y;
      m = fmaxf(m, rf[q]);
    }
    m = wave_max(m);
    double dd = 0.0;
#pragma unroll
    for (int q = 0; q < kThreads / 64; ++q) {
      if (ac[q] != ac[q]) dd += ac[q];
      else if (rf[q] != -INFINITY) dd += static_cast<double>(ac[q]) * static_cast<double>(__builtin_amdgcn_exp2f(rf[q] - m));
    }
    dd = wave_sum(dd);
    if (c.lane == 0) {
      const int row = fused_row_index<E, K>(a, b, r);
      uint64_t* rec = reinterpret_cast<uint64_t*>(const_cast<RowStat*>(a.stats) + static_cast<int64_t>(row) * c.G + c.g);
      st_agent(rec, static_cast<uint64_t>(__float_as_uint(m)));
      st_agent(rec + 1, dd != dd ? 0x7FF8000000000000ull : static_cast<uint64_t>(__double_as_longlong(dd)));
    }
  }
}

// Park the pair rows of a batch row (and its decision inputs) in LDS for its
// overlap stage.
template <class E, int K>
__device__ __forceinline__ void fused_park(const FusedCtx<E, K>& c, const FusedUnit<E, K>& u) {
  FusedShared<E, K>& sh = *c.sh;
#pragma unroll
  for (int i = 0; i < K; ++i)
#pragma unroll
    for (int j = 0; j < kFusedNV; ++j) {
      sh.pbuf[i][j][c.tid] = u.w[i][j];
      sh.pbuf[K + i][j][c.tid] = u.w[K + 1 + i][j];
    }
  if (c.tid < K) sh.pgx[c.tid] = u.gx;
  if (c.tid == 0) {
    sh.pb = u.b;
    sh.pT = u.T;
  }
}

// Stage 3: the group's records of every row (published one step earlier),
// the row normalisers in combine_row's order, the decision, and the overlap
// and residual sums of the slice from the parked rows.
template <class E, int K>
__device__ __forceinline__ void fused_pairs(const FusedCtx<E, K>& c, int b, const FusedPoll<K>& pl) {
  constexpr int EPV = E::EPV;
  constexpr int R = 2 * K + 1;
  const VerifyArgs& a = c.a;
  const int G = c.G, lane = c.lane;
  FusedShared<E, K>& sh = *c.sh;
#pragma unroll
  for (int i = 0; i < FusedPoll<K>::RW; ++i) {
    const int r = c.wave + kWaves * i;
    if (r >= R) break;
    const int row = fused_row_index<E, K>(a, b, r);
    const uint64_t* rec = reinterpret_cast<const uint64_t*>(a.stats + static_cast<int64_t>(row) * G);
    // the first poll was issued at the start of the step; polls again only
    // for records not yet complete
    // (checked once outside the loop: inside it the wait for a poll covers
    // every load issued before it)
    uint64_t w0 = pl.w0[i], w1 = pl.w1[i];
    bool timed_out = false;
    if (!__all(lane >= G || (w0 != kRecordEmpty && w1 != kRecordEmpty))) {
      for (unsigned spin = 0;; ++spin) {
        if (sh.gave_up || spin >= c.spin_limit) {
          timed_out = true;
          sh.gave_up = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
        if (lane < G) {
          if (w0 == kRecordEmpty) w0 = ld_agent(rec + 2 * lane);
          if (w1 == kRecordEmpty) w1 = ld_agent(rec + 2 * lane + 1);
        }
        if (__all(lane >= G || (w0 != kRecordEmpty && w1 != kRecordEmpty))) break;
      }
    }
    const float mc = lane < G ? __uint_as_float(static_cast<uint32_t>(w0)) : -INFINITY;
    const double dc = lane < G ? __longlong_as_double(static_cast<long long>(w1)) : 0.0;
    const float M = wave_max(mc);
    double dsum = 0.0;
    if (lane < G) {
      if (dc != dc) dsum += dc;
      else if (mc != -INFINITY) dsum += dc * static_cast<double>(__builtin_amdgcn_exp2f(mc - M));
    }
    double D = wave_sum(dsum);
    if (timed_out) D = NAN;  // reported as a row data error
    if (lane == 0) {
      const RowNorm nn = make_norm(M, D);
      sh.dec.nrm[r] = nn;
      if (c.g == 0) a.norms[row] = nn;
    }
  }
  __syncthreads();
  if (c.wave == 0) {
    DraftGather gx{0, 0.f, 0.f, 0.0};
    if (lane < K) gx = sh.pgx[lane];
    const int n = decide_wave<E>(a, b, sh.dec, gx, sh.pT, c.g == 0);
    if (lane == 0) {
      sh.n = n;
      if (c.g == 0) a.decision[b] = n;
    }
  }
  __syncthreads();
  const int n = sh.n;
  if (n >= 0) {
    const float s = scale_of(sh.pT);
    float al[K];
    float zp = 0.f, sd = 0.f, qg = 0.f;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      al[i] = 0.f;
      if (a.overlap == nullptr && i != n) continue;
      const RowNorm nt = sh.dec.nrm[i], nd = sh.dec.nrm[K + 1 + i];
      if (i == n) {
        const ResidualRef rr = residual_ref(nt, nd, 0.0);
#pragma unroll
        for (int j = 0; j < kFusedNV; ++j) {
          float xt[EPV], xd[EPV];
          E::widen(sh.pbuf[i][j][c.tid], xt);
          E::widen(sh.pbuf[K + i][j][c.tid], xd);
#pragma unroll
          for (int k = 0; k < EPV; ++k) {
            const ElemPQ e = elem_pq(xt[k], xd[k], s, nt, nd, rr);
            al[i] += e.mn;
            zp += e.pos ? e.g : 0.f;
            sd += e.diff();
            qg += e.pos ? e.mn : 0.f;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < kFusedNV; ++j) {
          float xt[EPV], xd[EPV];
          E::widen(sh.pbuf[i][j][c.tid], xt);
          E::widen(sh.pbuf[K + i][j][c.tid], xd);
#pragma unroll
          for (int k = 0; k < EPV; ++k) al[i] += min_prob(xt[k], xd[k], s, nt, nd);
        }
      }
    }
    // K overlaps and three residual sums: float64 wave sums, then the four waves in order
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const double v = wave_sum(static_cast<double>(al[i]));
      if (lane == 0) sh.pr[c.wave][i] = v;
    }
    if (n < K) {
      const double v0 = wave_sum(static_cast<double>(zp));
      const double v1 = wave_sum(static_cast<double>(sd));
      const double v2 = wave_sum(static_cast<double>(qg));
      if (lane == 0) {
        sh.pr[c.wave][K] = v0;
        sh.pr[c.wave][K + 1] = v1;
        sh.pr[c.wave][K + 2] = v2;
      }
    }
    __syncthreads();
    if (c.tid < K) {
      PairStat o;
      double t[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int q = 0; q < kWaves; ++q) {
        t[0] += sh.pr[q][c.tid];
        if (c.tid == n) {
          t[1] += sh.pr[q][K];
          t[2] += sh.pr[q][K + 1];
          t[3] += sh.pr[q][K + 2];
        }
      }
      o.alpha = t[0]; o.Z = t[1]; o.Sd = t[2]; o.Qg = t[3];
      a.pairs[static_cast<int64_t>(b * K + c.tid) * G + c.g] = o;
    }
  }
}

// One step of the pipeline, its loads issued in the order they are waited
// for: the first poll of the records of row j - 1 (parked one step earlier,
// its records published then), the draft logits of row j, then the loads of
// the group's batch row j + 1 into `ld`; then reduce row j (`st`, loaded one
// step earlier), run the overlap stage of row j - 1 from the parked rows, and
// park row j.  Row j + 1's loads stay in flight all the while.
template <class E, int K>
__device__ __forceinline__ void fused_step(const FusedCtx<E, K>& c, int j, int grp, int NG, int B,
                                           FusedUnit<E, K>& ld, FusedUnit<E, K>& st) {
  FusedShared<E, K>& sh = *c.sh;
  const int pb = sh.pb;
  FusedPoll<K> pl;
  fused_poll<E, K>(c, pb, pl);
  fused_gather<E, K>(c, st);
  __builtin_amdgcn_sched_barrier(0);
  const int bl = grp + (j + 1) * NG;
  fused_load<E, K>(c, bl < B ? bl : -1, ld);
  __builtin_amdgcn_sched_barrier(0);
  if (st.b >= 0) fused_stats<E, K>(c, st);
  if (pb >= 0) fused_pairs<E, K>(c, pb, pl);
  __syncthreads();  // the parked rows, part[] and the shared state are rewritten below
  fused_park<E, K>(c, st);
  __syncthreads();
}

// Group k = blockIdx.x / G takes batch rows k, k + NG, k + 2 NG, ...; its
// member g = blockIdx.x % G owns slice g of every row.  Two register sets
// alternate (the loop is unrolled twice) between the batch row being loaded
// and the one being reduced; the row in its overlap stage waits in LDS.
template <class E, int K>
__global__ __launch_bounds__(kThreads) void verify_fused_kernel(VerifyArgs a, int G, int NG, unsigned spin_limit) {
  __shared__ FusedShared<E, K> sh;
  const int grp = static_cast<int>(blockIdx.x) / G, g = static_cast<int>(blockIdx.x) - grp * G;
  if (grp >= NG) return;
  const int tid = threadIdx.x;
  if (tid == 0) {
    sh.pb = -1;
    sh.gave_up = 0;
  }
  __syncthreads();
  const FusedCtx<E, K> c{a,         G,           g,   g * (kThreads * kFusedNV * E::EPV), tid, tid >> 6, tid & 63,
                         spin_limit, &sh, a.rows.temp_scalar};
  const int B = a.B;
  FusedUnit<E, K> u0, u1;
  fused_load<E, K>(c, grp < B ? grp : -1, u0);
  for (int j = 0;; j += 2) {
    if (u0.b < 0 && sh.pb < 0) break;
    fused_step<E, K>(c, j, grp, NG, B, u1, u0);
    if (u1.b < 0 && sh.pb < 0) break;
    fused_step<E, K>(c, j + 1, grp, NG, B, u0, u1);
  }
}

}  // namespace sv

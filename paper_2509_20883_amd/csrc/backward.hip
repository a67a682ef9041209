// Backward + row-sparse optimizer kernels of the sparse embedding step (gfx950).
//
// RecIS backward workflow: the embedding gradients and the offsets kept from
// the forward pass update the optimizer state and the parameters in the
// Blocks directly ("Backward Update"; SparseAdam-style optimizers update the
// touched rows only).  The gradient of a unique key is the sum over its
// occurrences of the upstream gradient row of the occurrence's bag (scaled
// by 1/len for mean pooling; one position's row for the padded copy).
//
// The forward wrote, per unique key, a contiguous segment of the occurrence
// list.  Two strategies reduce it, as the paper's reduction operators pick a
// mapping by conflict rate ("reduce easy" / "reduce hard"):
//   k_bwd_short       a key with <= kLong occurrences: one lane group sums
//                     its segment and, fused, applies the optimizer to its row
//                     (the row and its state are prefetched while the
//                     gradient rows are being read)
//   k_bwd_long        a hot key: its segment is cut into units (kUnit
//                     positions, more for the hottest keys so a key has at
//                     most kMaxUnits units), each XCD taking a contiguous
//                     eighth of them; each unit writes its partial sum row
//                     (no atomics)
//   k_bwd_long_finish one block per hot key sums the partial rows of its
//                     units in a fixed order and applies the optimizer
// Without the optimizer (lookup_pool_bwd) the same kernels write grad_unique.
#include "device_common.h"

#include <hip/hip_ext.h>

namespace rs {

// Sum of v over the LANES lanes of a lane group (every lane gets it).
template <int LANES>
__device__ inline float group_sum(float v) {
#pragma unroll
  for (int d = LANES / 2; d >= 1; d >>= 1) v += __shfl_xor(v, d, LANES);
  return v;
}

// Optimizer state of E consecutive elements [lane*E, lane*E + E) of a row,
// and the row's state scalar (row-wise optimizers).
template <typename WT, int E>
struct RowFrag {
  float w[E], s1[E], s2[E], sr;
  __device__ inline void load(const uint8_t* row, int lane, int dim, int nstate, int rowscalar) {
    load_vals<WT, E>(reinterpret_cast<const WT*>(row) + lane * E, w);
    const float* base = reinterpret_cast<const float*>(row + static_cast<int64_t>(dim) * sizeof(WT));
    if (nstate >= 1) load_vals<float, E>(base + lane * E, s1);
    if (nstate == 2) load_vals<float, E>(base + dim + lane * E, s2);
    sr = rowscalar ? base[nstate * dim] : 0.f;  // the same word for the whole lane group
  }
  // Adagrad: acc += g^2; w -= lr g / (sqrt(acc) + eps).
  // Adam:    m = b1 m + (1-b1) g; v = b2 v + (1-b2) g^2; w -= lr (m/bc1) / (sqrt(v/bc2) + eps).
  // AdamW:   w -= (lr wd) w, then the Adam step.
  // Adam, epsilon-hat form: the same moments; w -= lr_t m / (sqrt(v) + eps).
  // Row-wise (ms = the row mean of g^2, summed over the lane group):
  //   Adagrad: acc += ms; w -= lr g / (sqrt(acc) + eps)
  //   Adam:    m per element as above; v = b2 v + (1-b2) ms per row;
  //            w -= lr (m/bc1) / (sqrt(v/bc2) + eps)
  // All lanes of the group call it together (the row-wise sum shuffles).
  template <int LANES>
  __device__ inline void update_store(uint8_t* row, int lane, int dim, const float (&g)[E], const OptArgs& o) {
    float* base = reinterpret_cast<float*>(row + static_cast<int64_t>(dim) * sizeof(WT));
    float* p = base + lane * E;
    if (o.opt >= 4) {
      float ss = 0.f;
#pragma unroll
      for (int k = 0; k < E; ++k) ss += g[k] * g[k];
      const float ms = group_sum<LANES>(ss) / static_cast<float>(dim);
      if (o.opt == 4) {
        sr = sr + ms;
        const float step = o.lr / (__builtin_sqrtf(sr) + o.eps);
#pragma unroll
        for (int k = 0; k < E; ++k) w[k] = w[k] - step * g[k];
        if (lane == 0) base[0] = sr;
      } else {
        sr = o.beta2 * sr + o.omb2 * ms;
        const float den = __builtin_sqrtf(sr / o.bc2) + o.eps;
#pragma unroll
        for (int k = 0; k < E; ++k) {
          s1[k] = o.beta1 * s1[k] + o.omb1 * g[k];
          w[k] = w[k] - o.lr * (s1[k] / o.bc1) / den;
        }
        store_vals_nt<float, E>(p, s1);
        if (lane == 0) base[dim] = sr;
      }
    } else if (o.opt == 0) {
#pragma unroll
      for (int k = 0; k < E; ++k) {
        s1[k] = s1[k] + g[k] * g[k];
        w[k] = w[k] - o.lr * g[k] / (__builtin_sqrtf(s1[k]) + o.eps);
      }
      store_vals_nt<float, E>(p, s1);
    } else {
#pragma unroll
      for (int k = 0; k < E; ++k) {
        s1[k] = o.beta1 * s1[k] + o.omb1 * g[k];
        s2[k] = o.beta2 * s2[k] + o.omb2 * g[k] * g[k];
        if (o.opt == 3) {
          w[k] = w[k] - o.lrt * s1[k] / (__builtin_sqrtf(s2[k]) + o.eps);
        } else {
          if (o.opt == 2) w[k] = w[k] - o.wdlr * w[k];
          w[k] = w[k] - o.lr * (s1[k] / o.bc1) / (__builtin_sqrtf(s2[k] / o.bc2) + o.eps);
        }
      }
      store_vals_nt<float, E>(p, s1);
      store_vals_nt<float, E>(p + dim, s2);
    }
    store_vals_nt<WT, E>(reinterpret_cast<WT*>(row) + lane * E, w);
  }
};

// Mean pooling's scale of gradient row (bag) r: 1 / the bag's length, from
// the forward's offsets (r < nref = bags; any other r contributes nothing).
__device__ inline float mean_scale(const Work& w, int r, uint32_t nref) {
  if (static_cast<uint32_t>(r) >= nref) return 0.f;
  const int64_t len = w.offsets[r + 1] - w.offsets[r];
  return 1.0f / static_cast<float>(max(len, int64_t(1)));
}

// Sum of the gradient rows of occurrence-list positions [p0, p0 + cnt),
// cnt <= kUnit.  The lanes of the group load the positions' gradient-row
// indices together (one round trip), share them by shuffles, and then read
// the gradient rows kBatch at a time.
template <typename GT, int E, int LANES, int MODE>
__device__ inline void sum_positions(const Work& w, const GT* __restrict__ grad, uint32_t nref, int p0, int cnt,
                                     int lane, float (&acc)[E]) {
  constexpr int D = LANES * E;
  constexpr int NR = (kUnit + LANES - 1) / LANES;  // positions per lane
  // gradient rows in flight: a small batch keeps more waves resident; narrow
  // rows (<= 4 lanes) take a whole unit's rows (128 values per lane) at once
  constexpr int kBatch = LANES <= 4 ? 128 / E : 8;
  int myref[NR];
  float mysc[NR];
#pragma unroll
  for (int k = 0; k < NR; ++k) {
    const int q = k * LANES + lane;
    myref[k] = q < cnt ? w.occ_ref[p0 + q] : -1;
  }
  if (MODE == 1) {
#pragma unroll
    for (int k = 0; k < NR; ++k) mysc[k] = mean_scale(w, myref[k], nref);
  }
#pragma unroll
  for (int q0 = 0; q0 < kUnit; q0 += kBatch) {
    if (q0 >= cnt) break;
    int ref[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int q = q0 + j;
      const int r = LANES > 1 ? __shfl(myref[q / LANES], q % LANES, LANES) : myref[q];
      ref[j] = q < cnt && static_cast<uint32_t>(r) < nref ? r : -1;
    }
    uint4 raw[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)  // every load issued before any is used
      raw[j] = ref[j] >= 0 ? load_raw16(grad + static_cast<int64_t>(ref[j]) * D + lane * E)
                           : make_uint4(0u, 0u, 0u, 0u);
    float x[kBatch][E];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) widen16<GT, E>(raw[j], x[j]);
    if (MODE == 1) {
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int q = q0 + j;
        const float sc = LANES > 1 ? __shfl(mysc[q / LANES], q % LANES, LANES) : mysc[q];
#pragma unroll
        for (int k = 0; k < E; ++k) x[j][k] *= sc;
      }
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
#pragma unroll
      for (int k = 0; k < E; ++k) acc[k] += x[j][k];
  }
}

// Sum of the gradient rows of K segments of the occurrence list
// ([st[k], st[k] + ct[k]), ct[k] <= kLong), taken as one sequence of at most
// K * kLong positions: the lanes load the positions' gradient-row indices
// together, share them by shuffles, and read the rows kBatch at a time, each
// added into its segment's accumulator.
template <typename GT, int E, int LANES, int MODE, int K>
__device__ inline void sum_segments(const Work& w, const GT* __restrict__ grad, uint32_t nref, const int (&st)[K],
                                    const int (&ct)[K], int lane, float (&acc)[K][E]) {
  constexpr int D = LANES * E;
  constexpr int MAXP = K * kLong;
  constexpr int NR = (MAXP + LANES - 1) / LANES;  // positions per lane
  constexpr int kBatch = 8;  // gradient rows in flight (111 VGPRs for fp32 rows: 4 waves per SIMD)
  int pre[K + 1];
  pre[0] = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) pre[k + 1] = pre[k] + ct[k];
  const int T = pre[K];
  int myref[NR];
  float mysc[NR];
#pragma unroll
  for (int j = 0; j < NR; ++j) {
    const int tq = j * LANES + lane;
    int kk = 0;
#pragma unroll
    for (int k = 1; k < K; ++k) kk += tq >= pre[k];
    const bool valid = tq < T;
    int sk = st[0], pk = 0;  // select, not a runtime index (keeps st / pre in registers)
#pragma unroll
    for (int k = 1; k < K; ++k)
      if (kk == k) {
        sk = st[k];
        pk = pre[k];
      }
    const int p = valid ? sk + (tq - pk) : 0;
    myref[j] = valid ? w.occ_ref[p] : -1;
  }
  if (MODE == 1) {
#pragma unroll
    for (int j = 0; j < NR; ++j) mysc[j] = mean_scale(w, myref[j], nref);
  }
#pragma unroll
  for (int q0 = 0; q0 < MAXP; q0 += kBatch) {
    if (q0 >= T) break;
    int ref[kBatch], kq[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int tq = q0 + j;
      const int r = LANES > 1 ? __shfl(myref[tq / LANES], tq % LANES, LANES) : myref[tq];
      ref[j] = tq < T && static_cast<uint32_t>(r) < nref ? r : -1;
      int kk = 0;
#pragma unroll
      for (int k = 1; k < K; ++k) kk += tq >= pre[k];
      kq[j] = kk;
    }
    uint4 raw[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)  // every load issued before any is used
      raw[j] = ref[j] >= 0 ? load_raw16(grad + static_cast<int64_t>(ref[j]) * D + lane * E)
                           : make_uint4(0u, 0u, 0u, 0u);
    float x[kBatch][E];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) widen16<GT, E>(raw[j], x[j]);
    if (MODE == 1) {
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int tq = q0 + j;
        const float sc = LANES > 1 ? __shfl(mysc[tq / LANES], tq % LANES, LANES) : mysc[tq];
#pragma unroll
        for (int e = 0; e < E; ++e) x[j][e] *= sc;
      }
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const bool hit = kq[j] == k;  // a select per accumulator, not an indexed access
#pragma unroll
        for (int e = 0; e < E; ++e) acc[k][e] += hit ? x[j][e] : 0.f;
      }
  }
}

// Keys with at most kLong occurrences: a lane group takes kShortKeys
// consecutive keys per iteration (their loads interleaved); block `blk` of
// `nblk` takes every nblk-th group of keys.
template <typename WT, typename GT, int LANES, int MODE, bool FUSED>
__device__ inline void bwd_short(const TableDev& t, const Work& w, uint32_t nref, const GT* __restrict__ grad, float* __restrict__ grad_unique, const OptArgs& o,
                                 int64_t blk, int64_t nblk) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  constexpr int GPB = kBlock / LANES;
  constexpr int D = LANES * E;
  constexpr int K = E == 4 ? kShortKeys : 1;  // bf16 gradient rows: one key (register budget)
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t U = w.scal[kCU];
  for (int64_t u0 = (blk * GPB + grp) * K; u0 < U; u0 += nblk * GPB * K) {
    Seg sg[K];
#pragma unroll
    for (int k = 0; k < K; ++k) sg[k] = w.useg[min(u0 + k, U - 1)];
    int st[K], ct[K];
    bool act[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      act[k] = u0 + k < U && sg[k].count <= kLong;  // hot keys: k_bwd_long
      st[k] = sg[k].start;
      ct[k] = act[k] ? sg[k].count : 0;
    }
    RowFrag<WT, E> fr[K];
    if (FUSED) {
#pragma unroll
      for (int k = 0; k < K; ++k)  // in flight while the gradients are read
        if (act[k] && sg[k].row >= 0) fr[k].load(t.store.row(sg[k].row), lane, D, t.nstate, t.rowscalar);
    }
    float acc[K][E];
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[k][e] = 0.f;
    sum_segments<GT, E, LANES, MODE, K>(w, grad, nref, st, ct, lane, acc);
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (!act[k]) continue;
      if (FUSED) {
        if (sg[k].row >= 0) fr[k].template update_store<LANES>(t.store.row(sg[k].row), lane, D, acc[k], o);
      } else {
        store_vals<float, E>(grad_unique + (u0 + k) * D + lane * E, acc[k]);
      }
    }
  }
}

// One lane group per backward unit of a hot key: the unit's partial sum is
// written to its own partial row.
template <typename GT, int LANES, int MODE>
__device__ inline void bwd_units(const Work& w, uint32_t nref, const GT* __restrict__ grad, int64_t blk,
                                 int64_t nblk) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  constexpr int GPB = kBlock / LANES;
  constexpr int D = LANES * E;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t units = w.scal[kCNUnits];
  for (int64_t unit = blk * GPB + grp; unit < units; unit += nblk * GPB) {
    const Unit un = w.units[unit];
    float acc[E];
#pragma unroll
    for (int q = 0; q < E; ++q) acc[q] = 0.f;
    for (int p = un.p0; p < un.p1; p += kUnit)
      sum_positions<GT, E, LANES, MODE>(w, grad, nref, p, min(kUnit, un.p1 - p), lane, acc);
    store_vals<float, E>(w.gpart + unit * D + lane * E, acc);
  }
}

// The two strategies run as consecutive launches (interleaving their blocks
// in one launch measured slower: the hot-key units' scattered gradient reads
// then compete with the short keys' row updates).
template <typename WT, typename GT, int LANES, int MODE, bool FUSED>
__global__ __launch_bounds__(kBlock) void k_bwd_short(TableDev t, Work w, uint32_t nref, const GT* __restrict__ grad, float* __restrict__ grad_unique,
                                                      OptArgs o) {
  bwd_short<WT, GT, LANES, MODE, FUSED>(t, w, nref, grad, grad_unique, o, blockIdx.x, gridDim.x);
}

template <typename GT, int LANES, int MODE>
__global__ __launch_bounds__(kBlock) void k_bwd_long(Work w, uint32_t nref, const GT* __restrict__ grad) {
  // XCD-contiguous: the dispatcher deals blocks to the 8 XCDs in turn, so
  // block b runs on XCD b % 8; XCD x takes the x-th eighth of the units that
  // exist (consecutive hot keys, so few features at a time: their gradient
  // rows are re-read from that XCD's L2).  Units are equal work (kUnit ids),
  // so the eighths balance.  The grid is a multiple of 8 blocks covering
  // every possible unit.
  const int64_t units = w.scal[kCNUnits];
  constexpr int64_t gpb = kBlock / LANES;
  const int64_t A = (units + gpb - 1) / gpb;  // blocks with units
  const int64_t per = (A + 7) / 8;
  const int64_t x = blockIdx.x % 8, i = blockIdx.x / 8;
  if (i >= per) return;
  const int64_t L = x * per + i;
  if (L >= A) return;
  bwd_units<GT, LANES, MODE>(w, nref, grad, L, 8 * per);
}

template <typename WT, int E, int LANES, bool FUSED>
__global__ __launch_bounds__(kBlock) void k_bwd_long_finish(TableDev t, Work w, float* __restrict__ grad_unique,
                                                            OptArgs o) {
  constexpr int GPB = kBlock / LANES;
  constexpr int D = LANES * E;
  __shared__ float red[GPB][D];
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t nlong = w.scal[kCNLong];
  for (int64_t li = blockIdx.x; li < nlong; li += gridDim.x) {
    const int u = w.long_u[li];
    const Seg sg = w.useg[u];
    const int nu = unit_count(sg.count);
    const int64_t u0 = w.long_start[li];
    RowFrag<WT, E> fr;
    uint8_t* rp = nullptr;
    if (FUSED && grp == 0 && sg.row >= 0) {
      rp = t.store.row(sg.row);
      fr.load(rp, lane, D, t.nstate, t.rowscalar);  // in flight while the partial rows are read
    }
    float acc[E];
#pragma unroll
    for (int q = 0; q < E; ++q) acc[q] = 0.f;
    for (int j = grp; j < nu; j += 2 * GPB) {
      float x[E], y[E];
      load_vals<float, E>(w.gpart + (u0 + j) * D + lane * E, x);
      const bool two = j + GPB < nu;
      if (two) load_vals<float, E>(w.gpart + (u0 + j + GPB) * D + lane * E, y);
#pragma unroll
      for (int q = 0; q < E; ++q) acc[q] += x[q];
      if (two) {
#pragma unroll
        for (int q = 0; q < E; ++q) acc[q] += y[q];
      }
    }
#pragma unroll
    for (int q = 0; q < E; ++q) red[grp][lane * E + q] = acc[q];
    __syncthreads();
    for (int h = GPB / 2; h >= 1; h >>= 1) {
      if (grp < h) {
#pragma unroll
        for (int q = 0; q < E; ++q) red[grp][lane * E + q] += red[grp + h][lane * E + q];
      }
      __syncthreads();
    }
    if (grp == 0) {
#pragma unroll
      for (int q = 0; q < E; ++q) acc[q] = red[0][lane * E + q];
      if (FUSED) {
        if (rp) fr.template update_store<LANES>(rp, lane, D, acc, o);
      } else {
        store_vals<float, E>(grad_unique + static_cast<int64_t>(u) * D + lane * E, acc);
      }
    }
    __syncthreads();  // red is reused by the block's next key
  }
}

// The occurrence list the backward reads: position occ_pos[i] of id i
// receives the gradient row the pool gave that id (id_ref).  Ids outside
// the pooled range [lo, hi) get no gradient row (-1); ids of a rejected key
// have no position.
//
// One block per dedup tile (kOccListNT threads, 4 ids each).  A record's ids
// in the tile hold the consecutive positions [base, base + count) of its
// key's segment, one per rank, so the block counting-sorts its ids by record
// in LDS (the tile's records are a contiguous range of its dedup block's
// list) and stores slot after slot: consecutive lanes write consecutive
// positions along each record's run, instead of one scattered 4-byte store
// per id.
constexpr int kOccListNT = kDedupTile / 4;

__global__ __launch_bounds__(kOccListNT) void k_occ_list(Work w, int64_t n) {
  constexpr int T = kDedupTile;
  __shared__ int cnt[T];  // per record of the tile: its ids, then its first slot
  __shared__ int spos[T], sref[T];
  __shared__ int wsh[kOccListNT / kWave + 1];
  __shared__ int rlo_sh;
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * T + threadIdx.x * 4;
  const int64_t lo = min(max(w.scal[kCIdLo], int64_t(0)), n);
  const int64_t hi = min(max(w.scal[kCIdHi], lo), n);
  uint32_t o[4];
  int pos[4], ref[4];
  if (i0 + 4 <= n) {
    const int4 ow = *reinterpret_cast<const int4*>(w.occ_word + i0);
    const int4 p = *reinterpret_cast<const int4*>(w.occ_pos + i0);
    const int4 r = *reinterpret_cast<const int4*>(w.id_ref + i0);
    o[0] = ow.x; o[1] = ow.y; o[2] = ow.z; o[3] = ow.w;
    pos[0] = p.x; pos[1] = p.y; pos[2] = p.z; pos[3] = p.w;
    ref[0] = r.x; ref[1] = r.y; ref[2] = r.z; ref[3] = r.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool v = i0 + k < n;
      o[k] = v ? w.occ_word[i0 + k] : kOccRejected;
      pos[k] = v ? w.occ_pos[i0 + k] : -1;
      ref[k] = v ? w.id_ref[i0 + k] : -1;
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (i0 + k < lo || i0 + k >= hi) ref[k] = -1;
    if (pos[k] < 0) o[k] = kOccRejected;  // no list entry
  }
  // the tile's first record
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    cnt[threadIdx.x * 4 + k] = 0;
    spos[threadIdx.x * 4 + k] = -1;  // a slot no id fills is skipped
  }
  if (threadIdx.x == 0) rlo_sh = 0x7FFFFFFF;
  __syncthreads();
  int m = 0x7FFFFFFF;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (o[k] != kOccRejected) m = min(m, static_cast<int>(o[k] >> 12));
  if (m != 0x7FFFFFFF) atomicMin(&rlo_sh, m);
  __syncthreads();
  const int rlo = rlo_sh;
  // ids per record, then each record's first slot (exclusive scan)
  int d[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    d[k] = o[k] == kOccRejected ? -1 : static_cast<int>(o[k] >> 12) - rlo;
    if (d[k] >= T) d[k] = -1;  // outside the tile's records: cannot happen, stored directly below
    if (d[k] >= 0) atomicAdd(&cnt[d[k]], 1);
  }
  __syncthreads();
  int c4[4], sum = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    c4[k] = cnt[threadIdx.x * 4 + k];
    sum += c4[k];
  }
  int total;
  int ex = block_excl_scan<kOccListNT>(sum, wsh, total);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    cnt[threadIdx.x * 4 + k] = ex;
    ex += c4[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (pos[k] < 0) continue;
    const int slot = d[k] >= 0 ? cnt[d[k]] + static_cast<int>(o[k] & 0xFFFu) : T;
    if (slot < T) {
      spos[slot] = pos[k];
      sref[slot] = ref[k];
    } else {
      w.occ_ref[pos[k]] = ref[k];
    }
  }
  __syncthreads();
  for (int s = threadIdx.x; s < min(total, T); s += kOccListNT) {
    const int p = spos[s];
    if (p < 0) continue;
    w.occ_ref[p] = sref[s];
  }
}

template <typename WT, typename GT, int LANES, int MODE, bool FUSED>
static hipError_t bwd_launch(const TableDev& t, const Work& w, uint32_t nref, int64_t n, const void* grad,
                             float* gu, const OptArgs& o, hipEvent_t* ev_s, hipEvent_t* ev_l, hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  constexpr int GPB = kBlock / LANES;
  const GT* g = static_cast<const GT*>(grad);
  // grid-stride loops over device-side counts (U, units, hot keys): a grid
  // of at most kResident blocks per strategy keeps every CU busy without
  // dispatching wavefronts that would find no work
  // optional timing events are timestamped by the dispatches themselves
  // (short keys: their kernel; hot keys: unit sums start to finish end)
  hipEvent_t s0 = ev_s ? ev_s[0] : nullptr, s1 = ev_s ? ev_s[1] : nullptr;
  hipEvent_t l0 = ev_l ? ev_l[0] : nullptr, l1 = ev_l ? ev_l[1] : nullptr;
  hipExtLaunchKernelGGL((k_bwd_short<WT, GT, LANES, MODE, FUSED>), dim3(grid_for(n, GPB, kResident)), dim3(kBlock), 0,
                        s, s0, s1, 0, t, w, nref, g, gu, o);
  // one lane group per possible unit (the device-side count is at most
  // 2n/kUnit + 2): no group takes a second unit while others are idle
  hipExtLaunchKernelGGL((k_bwd_long<GT, LANES, MODE>), dim3((grid_for(2 * (n / kUnit) + 2, GPB) + 7) / 8 * 8),
                        dim3(kBlock), 0, s,
                        l0, nullptr, 0, w, nref, g);
  hipExtLaunchKernelGGL((k_bwd_long_finish<WT, E, LANES, FUSED>), dim3(grid_for(n / kLong + 1, 1, 4 * kResident)),
                        dim3(kBlock), 0, s, nullptr, l1, 0, t, w, gu, o);
  return hipGetLastError();
}

template <typename WT, typename GT, int MODE, bool FUSED>
static hipError_t bwd_dim(const TableDev& t, const Work& w, uint32_t nref, int64_t n, const void* grad,
                          float* gu, const OptArgs& o, hipEvent_t* es, hipEvent_t* el, hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  switch (t.dim / E) {
    case 1: return bwd_launch<WT, GT, 1, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 2: return bwd_launch<WT, GT, 2, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 4: return bwd_launch<WT, GT, 4, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 8: return bwd_launch<WT, GT, 8, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 16: return bwd_launch<WT, GT, 16, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 32: return bwd_launch<WT, GT, 32, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    case 64: return bwd_launch<WT, GT, 64, MODE, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename WT, bool FUSED>
static hipError_t bwd_mode(const TableDev& t, const Work& w, uint32_t nref, int64_t n, int mode,
                           const void* grad, float* gu, const OptArgs& o, hipEvent_t* es, hipEvent_t* el,
                           hipStream_t s) {
  if (mode == 2 || mode == 3) return bwd_dim<WT, WT, 0, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
  if (mode == 1) return bwd_dim<WT, float, 1, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
  return bwd_dim<WT, float, 0, FUSED>(t, w, nref, n, grad, gu, o, es, el, s);
}

hipError_t launch_bwd(const TableDev& t, const Work& w, int64_t nref, int64_t n, int mode, const void* grad,
                      float* grad_unique, const OptArgs* opt, hipEvent_t* ev_list, hipEvent_t* ev_short,
                      hipEvent_t* ev_long, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  {
    hipEvent_t e0 = ev_list ? ev_list[0] : nullptr, e1 = ev_list ? ev_list[1] : nullptr;
    const dim3 grid(static_cast<unsigned>((n + kDedupTile - 1) / kDedupTile));
    hipExtLaunchKernelGGL(k_occ_list, grid, dim3(kOccListNT), 0, s, e0, e1, 0, w, n);
  }
  const OptArgs o = opt ? *opt : OptArgs{0, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 1.f, 1.f, 0.f, 0.f};
  if (opt)
    return t.row_dtype ? bwd_mode<uint16_t, true>(t, w, static_cast<uint32_t>(nref), n, mode, grad, grad_unique, o, ev_short, ev_long, s)
                       : bwd_mode<float, true>(t, w, static_cast<uint32_t>(nref), n, mode, grad, grad_unique, o, ev_short, ev_long, s);
  return t.row_dtype ? bwd_mode<uint16_t, false>(t, w, static_cast<uint32_t>(nref), n, mode, grad, grad_unique, o, ev_short, ev_long, s)
                     : bwd_mode<float, false>(t, w, static_cast<uint32_t>(nref), n, mode, grad, grad_unique, o, ev_short, ev_long, s);
}

// ---------------------------------------------------------------------------
// optimizer from a written grad_unique (the two-call path)
// ---------------------------------------------------------------------------

template <typename WT, int LANES>
__global__ __launch_bounds__(kBlock) void k_opt(TableDev t, Work w, const float* __restrict__ grad_unique, OptArgs o) {
  constexpr int E = 4;
  constexpr int GPB = kBlock / LANES;
  constexpr int D = LANES * E;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t U = w.scal[kCU];
  for (int64_t u = static_cast<int64_t>(blockIdx.x) * GPB + grp; u < U; u += static_cast<int64_t>(gridDim.x) * GPB) {
    const int64_t r = w.useg[u].row;
    if (r < 0) continue;
    uint8_t* rp = t.store.row(r);
    RowFrag<WT, E> fr;
    fr.load(rp, lane, D, t.nstate, t.rowscalar);
    float g[E];
    load_vals<float, E>(grad_unique + u * D + lane * E, g);
    fr.template update_store<LANES>(rp, lane, D, g, o);
  }
}

template <typename WT>
static hipError_t opt_dim(const TableDev& t, const Work& w, int64_t n, const float* gu, const OptArgs& o,
                          hipStream_t s) {
  switch (t.dim / 4) {
    case 2: k_opt<WT, 2><<<grid_for(n, kBlock / 2, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    case 4: k_opt<WT, 4><<<grid_for(n, kBlock / 4, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    case 8: k_opt<WT, 8><<<grid_for(n, kBlock / 8, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    case 16: k_opt<WT, 16><<<grid_for(n, kBlock / 16, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    case 32: k_opt<WT, 32><<<grid_for(n, kBlock / 32, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    case 64: k_opt<WT, 64><<<grid_for(n, kBlock / 64, kResident), kBlock, 0, s>>>(t, w, gu, o); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_opt(const TableDev& t, const Work& w, int64_t n, const float* grad_unique, const OptArgs& opt,
                      hipEvent_t* ev, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (ev && ev[0]) (void)hipEventRecord(ev[0], s);
  const hipError_t e =
      t.row_dtype ? opt_dim<uint16_t>(t, w, n, grad_unique, opt, s) : opt_dim<float>(t, w, n, grad_unique, opt, s);
  if (ev && ev[1]) (void)hipEventRecord(ev[1], s);
  return e;
}

}  // namespace rs

// Forward gather + pool kernels of the sparse embedding step (gfx950).
//
// RecIS forward workflow: one IDMap lookup per id gives the offset, the row
// is read at that offset and the rows of a bag are reduced (sum, mean) or
// copied into a padded sequence ("Forward Pass", "Reduction Operations",
// "Gather").  The lookup happened in the dedup passes, which also gave every
// occurrence its row (occ_row); these kernels read each occurrence's row
// with 16-byte vector loads, one lane group of D*sizeof(row)/16 lanes per
// row, and write the gradient row of each id (id_ref, in id order), from
// which the backward builds its occurrence list.
//
// A lane group handles one bag per lane and requests 16 rows of them at a
// time, for single-id and long bags alike.
#include "device_common.h"

#include <hip/hip_ext.h>

namespace rs {


typedef float f32x4 __attribute__((ext_vector_type(4)));

// The ids the bags cover, [offsets[0], offsets[bags]) clamped to [0, n]: the
// backward gives ids outside it no gradient row.
__device__ inline void record_pooled_range(const Work& w, const int64_t* offsets, int64_t n, int64_t bags) {
  const int64_t lo = min(max(offsets[0], int64_t(0)), n);
  w.scal[kCIdLo] = lo;
  w.scal[kCIdHi] = min(max(offsets[bags], lo), n);
}

// acc += the E row elements held raw in v (16 bytes of the row)
template <typename WT, int E>
__device__ inline void add_raw(float (&acc)[E], const uint4& v);
template <>
__device__ inline void add_raw<float, 4>(float (&acc)[4], const uint4& v) {
  acc[0] += __uint_as_float(v.x);
  acc[1] += __uint_as_float(v.y);
  acc[2] += __uint_as_float(v.z);
  acc[3] += __uint_as_float(v.w);
}
template <>
__device__ inline void add_raw<uint16_t, 8>(float (&acc)[8], const uint4& v) {
  const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    acc[2 * k] += __uint_as_float(u[k] << 16);
    acc[2 * k + 1] += __uint_as_float(u[k] & 0xFFFF0000u);
  }
}

// Inclusive scan of v over the LANES lanes of a lane group.
template <int LANES>
__device__ inline int64_t group_incl_scan(int64_t v, int lane) {
#pragma unroll
  for (int d = 1; d < LANES; d <<= 1) {
    const int64_t t = __shfl_up(v, d, LANES);
    if (lane >= d) v += t;
  }
  return v;
}

// A lane group of LANES lanes pools LANES consecutive bags (lane q owns bag
// g0 + q).  Their positions, taken as one sequence, are read in chunks of C:
// the lanes load the chunk's occurrence rows and list positions (J per
// lane), the next chunk's are requested before this chunk's rows are used,
// and all C rows of a chunk are requested before any is added -- C rows in
// flight whether the bags hold one id or hundreds.  The rows are then added
// in order into one running accumulator; a cursor over the bags' cumulative
// lengths flushes a bag (one non-temporal row store) when the sequence passes
// its end, so empty bags are flushed as zeros and no per-bag accumulators
// are held.  The walk also writes each id's gradient row (its bag).
// For well-formed offsets (each bag starts where the previous one ends) the
// sequence is positions offsets[g0] ... ; malformed offsets give wrong
// sums, never an access outside [0, n).
template <typename WT, int LANES, int MODE, int C>
__global__ __launch_bounds__(kBlock) void k_pool(TableDev t, Work w, const int64_t* __restrict__ offsets, int64_t n,
                                                 int64_t bags, float* __restrict__ out) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  constexpr int D = LANES * E;
  constexpr int GPB = kBlock / LANES;
  constexpr int J = (C + LANES - 1) / LANES;  // chunk positions per lane
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  if (blockIdx.x == 0 && threadIdx.x == 0) record_pooled_range(w, offsets, n, bags);
  const int64_t g0 = (static_cast<int64_t>(blockIdx.x) * GPB + grp) * LANES;
  if (g0 >= bags) return;
  const int nb = static_cast<int>(min(static_cast<int64_t>(LANES), bags - g0));
  // this lane's bag, CSR bounds clamped to [0, n]; positions fit 32 bits (n <= 2^28)
  const int n32 = static_cast<int>(n);
  const int64_t gq = g0 + min(lane, nb - 1);
  const int bq = min(max(static_cast<int>(offsets[gq]), 0), n32);
  const int eq = min(max(static_cast<int>(offsets[gq + 1]), bq), n32);
  const int len = lane < nb ? eq - bq : 0;
  const int64_t cum = group_incl_scan<LANES>(len, lane);  // end of bag `lane` in the sequence
  // at most n ids for well-formed offsets (malformed ones are cut there)
  const int total = static_cast<int>(min(__shfl(cum, LANES - 1, LANES), static_cast<int64_t>(n32)));
  const int p0 = __shfl(bq, 0, LANES);                     // the sequence starts at the first bag's start
  int64_t rr[J];
  auto load_idx = [&](int t0) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = lane + j * LANES;
      const bool valid = c < C && t0 + c < total;
      const int p = valid ? min(p0 + t0 + c, n32 - 1) : 0;  // total > 0: position 0 exists
      rr[j] = w.occ_row[p];
      if (!valid) rr[j] = -1;
    }
  };
  float acc[E];
#pragma unroll
  for (int k = 0; k < E; ++k) acc[k] = 0.f;
  int q = 0;                                   // the bag the running sum belongs to (< nb)
  int64_t cq = __shfl(cum, 0, LANES);          // its end
  int64_t bstart = 0;                          // its start
  auto flush = [&]() {
    // the pooled output is streamed out once: non-temporal stores
    const int64_t blen = cq - bstart;
    if (MODE == 1 && blen > 0) {
      const float l = static_cast<float>(blen);
#pragma unroll
      for (int k = 0; k < E; ++k) acc[k] = acc[k] / l;
    }
    float* op = out + (g0 + q) * D + lane * E;
#pragma unroll
    for (int k = 0; k < E; k += 4) {
      const f32x4 v = {acc[k], acc[k + 1], acc[k + 2], acc[k + 3]};
      __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(op + k));
    }
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] = 0.f;
    ++q;
    bstart = cq;
    cq = __shfl(cum, min(q, LANES - 1), LANES);
  };
  if (total > 0) load_idx(0);
  for (int t0 = 0; t0 < total; t0 += C) {
    uint4 x[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int64_t r = LANES > 1 ? __shfl(rr[c / LANES], c % LANES, LANES) : rr[c];
      x[c] = make_uint4(0u, 0u, 0u, 0u);
      if (r >= 0) x[c] = *reinterpret_cast<const uint4*>(t.store.row(r) + lane * 16);
    }
    if (t0 + C < total) load_idx(t0 + C);  // the next chunk's row ids replace rr
    int myq[J];  // bag of this lane's positions in the chunk
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int tt = t0 + c;
      if (tt >= total) break;
      while (q < nb && tt >= cq) flush();  // bags ending before this id (empty ones flush zeros)
      if (lane == c % LANES) myq[c / LANES] = q;
      add_raw<WT, E>(acc, x[c]);
    }
    // each id of the chunk: the gradient row it reads in the backward (its
    // bag); consecutive lanes write consecutive ids (plain stores: a narrow
    // lane group writes only 16 bytes per chunk, which the L2 merges)
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = lane + j * LANES;
      if (c >= C || t0 + c >= total || p0 + t0 + c >= n32) continue;
      w.id_ref[p0 + t0 + c] = static_cast<int>(g0 + myq[j]);
    }
  }
  while (q < nb) flush();  // the last bag and any empty bags after it
}

// Padded copy: block = (bag, TCH positions); a lane group copies TCH / groups
// positions, with their loads issued together.
template <typename WT, int LANES>
__global__ __launch_bounds__(kBlock) void k_pool_none(TableDev t, Work w, const int64_t* __restrict__ offsets,
                                                      int64_t n, int64_t bags, int64_t L, bool tail,
                                                      WT* __restrict__ out, uint8_t* __restrict__ mask) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  constexpr int D = LANES * E;
  constexpr int GPB = kBlock / LANES;
  constexpr int TCH = GPB > 64 ? GPB : 64;  // positions per block
  constexpr int K = TCH / GPB;               // positions per lane group
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  if (blockIdx.x == 0 && threadIdx.x == 0) record_pooled_range(w, offsets, n, bags);
  const int64_t nch = (L + TCH - 1) / TCH;
  for (int64_t blk = blockIdx.x; blk < bags * nch; blk += gridDim.x) {
    const int64_t g = blk / nch, c = blk % nch;
    const int64_t b = min(max(offsets[g], int64_t(0)), n);
    const int64_t len = min(max(offsets[g + 1], b), n) - b;
    // the copied window: ids [skip, skip + min(len, L)) of the bag
    const int64_t skip = tail && len > L ? len - L : 0;
    int64_t tp[K], r[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      tp[k] = c * TCH + grp + k * GPB;
      const bool act = tp[k] < L && tp[k] < len;
      r[k] = act ? w.occ_row[b + skip + tp[k]] : -1;
    }
    uint4 v[K];
#pragma unroll
    for (int k = 0; k < K; ++k)
      v[k] = r[k] >= 0 ? *reinterpret_cast<const uint4*>(reinterpret_cast<const WT*>(t.store.row(r[k])) + lane * E)
                       : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (tp[k] >= L) continue;
      *reinterpret_cast<uint4*>(out + (g * L + tp[k]) * D + lane * E) = v[k];
      if (lane == 0) {
        mask[g * L + tp[k]] = tp[k] < len ? 1 : 0;
        if (tp[k] < len) w.id_ref[b + skip + tp[k]] = static_cast<int>(g * L + tp[k]);
      }
    }
    if (c == 0 && lane == 0) {
      // ids outside the window (past L, or before skip): in the occurrence
      // list (the key is touched) but without a gradient row
      const int64_t x0 = tail ? 0 : L, x1 = tail ? skip : len;
      for (int64_t tpos = x0 + grp; tpos < x1; tpos += GPB) w.id_ref[b + tpos] = -1;
    }
  }
}

// The launch takes optional start / stop events that the dispatch itself
// timestamps (the kernel's own execution, no extra packets on the stream).
template <typename WT, int LANES>
static hipError_t pool_mode(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags,
                            int mode, int64_t pad_len, void* out, uint8_t* mask, hipEvent_t e0, hipEvent_t e1,
                            hipStream_t s) {
  constexpr int GPB = kBlock / LANES;
  if (mode == 2 || mode == 3) {
    constexpr int TCH = GPB > 64 ? GPB : 64;
    const int64_t nch = (pad_len + TCH - 1) / TCH;
    hipExtLaunchKernelGGL((k_pool_none<WT, LANES>), dim3(grid_for(bags * nch, 1, 1 << 20)), dim3(kBlock), 0, s, e0, e1,
                          0, t, w, offsets, n, bags, pad_len, mode == 3, static_cast<WT*>(out), mask);
  } else {
    // one lane group per LANES bags (one bag per lane), 16 rows in flight
    float* o = static_cast<float*>(out);
    const unsigned g = grid_for(bags, static_cast<int64_t>(GPB) * LANES, int64_t(1) << 31);
    if (mode == 1)
      hipExtLaunchKernelGGL((k_pool<WT, LANES, 1, 16>), dim3(g), dim3(kBlock), 0, s, e0, e1, 0, t, w, offsets, n, bags,
                            o);
    else
      hipExtLaunchKernelGGL((k_pool<WT, LANES, 0, 16>), dim3(g), dim3(kBlock), 0, s, e0, e1, 0, t, w, offsets, n, bags,
                            o);
  }
  return hipGetLastError();
}

template <typename WT>
static hipError_t pool_dim(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags, int mode,
                           int64_t pad_len, void* out, uint8_t* mask, hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  switch (t.dim / E) {
    case 1: return pool_mode<WT, 1>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 2: return pool_mode<WT, 2>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 4: return pool_mode<WT, 4>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 8: return pool_mode<WT, 8>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 16: return pool_mode<WT, 16>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 32: return pool_mode<WT, 32>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    case 64: return pool_mode<WT, 64>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_pool(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags, int mode,
                       int64_t pad_len, void* out, uint8_t* mask, hipEvent_t* ev, hipStream_t s) {
  if (bags <= 0) return hipSuccess;
  hipEvent_t e0 = ev ? ev[0] : nullptr, e1 = ev ? ev[1] : nullptr;
  const hipError_t e = t.row_dtype ? pool_dim<uint16_t>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s)
                                   : pool_dim<float>(t, w, offsets, n, bags, mode, pad_len, out, mask, e0, e1, s);
  return e;
}

}  // namespace rs

// HIP kernels of the sparse embedding step for gfx950 (CDNA4).
//
// Step (RecIS, "Optimization for Memory Bound" — two-tier IDMap + Blocks
// store and its forward / backward workflow):
//   dedup        k_dedup_local -> k_flag_count -> k_scan_small -> k_compact -> k_inverse
//   segments     k_tile_reduce -> k_scan_small -> k_seg_apply (also clears the dedup scratch)
//   IDMap        k_idmap_probe -> k_tile_reduce -> k_scan_small -> k_idmap_insert (row init)
//   forward      k_pool / k_pool_none: gather + sum / mean / padded copy, and the
//                occurrence list of every unique id for the backward
//   backward     k_bwd_chunks (+ fused optimizer) -> k_bwd_straddle
//   optimizer    k_opt (when the backward writes grad_unique instead)
//
// Every hot kernel moves rows with 16-byte vector loads / stores, one lane
// group per row (row bytes / 16 lanes), so a 64-lane wavefront has 4..16 rows
// in flight ("Vectorized Memory Access").  Reductions avoid global atomics on
// hot keys: occurrences of a key are pre-merged in LDS per tile during dedup
// ("Atomic Operation Optimization"), and the backward reads a per-key
// occurrence list cut into fixed chunks, so a hot key is spread over many lane
// groups instead of serialising on one address.
#include "rs_internal.h"

namespace rs {

// ---------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// Round to nearest, ties to even; NaN -> 0x7FC0.
__device__ inline uint16_t f32_to_bf16(float x) {
  const uint32_t b = __float_as_uint(x);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu) != 0u) return 0x7FC0;
  return static_cast<uint16_t>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__device__ inline int wave_incl_scan(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

__device__ inline int wave_sum(int v) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, kWave);
  return v;
}

// Exclusive block scan of one int per thread; `sh` holds NT/64 + 1 ints.
template <int NT>
__device__ inline int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const int inc = wave_incl_scan(v);
  if (lane == kWave - 1) sh[wid] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < NT / kWave; ++w) {
      const int t = sh[w];
      sh[w] = run;
      run += t;
    }
    sh[NT / kWave] = run;
  }
  __syncthreads();
  const int ex = sh[wid] + inc - v;
  total = sh[NT / kWave];
  __syncthreads();
  return ex;
}

template <int NT>
__device__ inline int block_sum(int v, int* sh) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  v = wave_sum(v);
  if (lane == 0) sh[wid] = v;
  __syncthreads();
  int t = 0;
  if (threadIdx.x == 0)
    for (int w = 0; w < NT / kWave; ++w) t += sh[w];
  return t;  // valid in thread 0
}

// 8 consecutive int32 starting at p[i0] (i0 % 8 == 0), zero past n.
__device__ inline void load8(const int32_t* __restrict__ p, int64_t i0, int64_t n, int (&v)[8]) {
  if (i0 + 8 <= n) {
    const int4 a = *reinterpret_cast<const int4*>(p + i0);
    const int4 b = *reinterpret_cast<const int4*>(p + i0 + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = (i0 + k < n) ? p[i0 + k] : 0;
  }
}

// E fp32 values from a 16-byte-aligned row fragment of type T (f32 or bf16).
template <typename T, int E>
__device__ inline void load_vals(const T* __restrict__ p, float (&v)[E]);

template <>
__device__ inline void load_vals<float, 4>(const float* __restrict__ p, float (&v)[4]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
template <>
__device__ inline void load_vals<float, 8>(const float* __restrict__ p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ inline void load_vals<uint16_t, 8>(const uint16_t* __restrict__ p, float (&v)[8]) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(w[k] << 16);
    v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
  }
}
template <>
__device__ inline void load_vals<uint16_t, 4>(const uint16_t* __restrict__ p, float (&v)[4]) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(a.x << 16);
  v[1] = __uint_as_float(a.x & 0xFFFF0000u);
  v[2] = __uint_as_float(a.y << 16);
  v[3] = __uint_as_float(a.y & 0xFFFF0000u);
}

template <typename T, int E>
__device__ inline void store_vals(T* __restrict__ p, const float (&v)[E]);

template <>
__device__ inline void store_vals<float, 4>(float* __restrict__ p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
template <>
__device__ inline void store_vals<float, 8>(float* __restrict__ p, const float (&v)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ inline void store_vals<uint16_t, 8>(uint16_t* __restrict__ p, const float (&v)[8]) {
  uint4 a;
  a.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  a.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  a.z = static_cast<uint32_t>(f32_to_bf16(v[4])) | (static_cast<uint32_t>(f32_to_bf16(v[5])) << 16);
  a.w = static_cast<uint32_t>(f32_to_bf16(v[6])) | (static_cast<uint32_t>(f32_to_bf16(v[7])) << 16);
  *reinterpret_cast<uint4*>(p) = a;
}
template <>
__device__ inline void store_vals<uint16_t, 4>(uint16_t* __restrict__ p, const float (&v)[4]) {
  uint2 a;
  a.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  a.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  *reinterpret_cast<uint2*>(p) = a;
}

inline unsigned grid_for(int64_t work_items, int64_t per_block, int64_t cap = 1 << 20) {
  int64_t g = (work_items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g);
}

// Insert an encoded key into the IDMap (linear probing); returns the slot or -1.
__device__ inline int64_t idmap_claim(const TableDev& t, unsigned long long e) {
  uint64_t h = idmap_hash(e) & t.cap_mask;
  for (uint64_t probe = 0; probe <= t.cap_mask; ++probe) {
    const unsigned long long old = atomicCAS(&t.slots[h].key, kEncEmpty, e);
    if (old == kEncEmpty || old == e) return static_cast<int64_t>(h);
    h = (h + 1) & t.cap_mask;
  }
  return -1;
}

// Find an encoded key; returns its row, or -1 when an empty slot ends the probe.
__device__ inline int64_t idmap_lookup(const TableDev& t, unsigned long long e) {
  uint64_t h = idmap_hash(e) & t.cap_mask;
  for (uint64_t probe = 0; probe <= t.cap_mask; ++probe) {
    const Slot sl = t.slots[h];
    if (sl.key == e) return sl.row;
    if (sl.key == kEncEmpty) return -1;
    h = (h + 1) & t.cap_mask;
  }
  return -1;
}

// ---------------------------------------------------------------------------
// generic scalar / fill kernels
// ---------------------------------------------------------------------------

__global__ void k_fill_u64(unsigned long long* p, unsigned long long v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

hipError_t launch_fill_u64(unsigned long long* p, unsigned long long v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_fill_u64<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(p, v, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// dedup (unique keys in first-occurrence order + inverse index)
// ---------------------------------------------------------------------------

// Pass 1: a tile of kDedupTile occurrences is deduplicated in an LDS hash
// table; each distinct key of the tile then does ONE global insert into the
// scratch table: atomicMin of its first position, atomicAdd of its count.
// The value returned by that atomicAdd is the tile's base rank among the
// key's occurrences, so every occurrence also learns its rank (occ_rank),
// which later places it in the key's occurrence list without more atomics.
__global__ __launch_bounds__(kBlock) void k_dedup_local(const int64_t* __restrict__ values, int64_t n,
                                                        Scratch sc, int32_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ occ_rank, int* err) {
  __shared__ unsigned long long lkey[kDedupLdsSlots];
  __shared__ unsigned int lmin[kDedupLdsSlots];
  __shared__ unsigned int lcnt[kDedupLdsSlots];
  __shared__ int lgs[kDedupLdsSlots];
  __shared__ unsigned int lbase[kDedupLdsSlots];
  const int tid = threadIdx.x;
  for (int s = tid; s < kDedupLdsSlots; s += kBlock) {
    lkey[s] = kEncEmpty;
    lmin[s] = 0xFFFFFFFFu;
    lcnt[s] = 0u;
  }
  __syncthreads();
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kDedupTile;
  int ls[kDedupItems];
  unsigned int lr[kDedupItems];
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) {
    const int64_t i = base + k * kBlock + tid;
    ls[k] = -1;
    lr[k] = 0;
    if (i < n) {
      const unsigned long long e = static_cast<unsigned long long>(values[i]) ^ kSign;
      if (e <= kEncTomb) {
        atomicOr(err, kErrKey);
      } else {
        unsigned int h = static_cast<unsigned int>(mix64(e) >> 40) & (kDedupLdsSlots - 1);
        while (true) {  // at most kDedupTile keys in 2x slots: an empty slot always exists
          const unsigned long long old = atomicCAS(&lkey[h], kEncEmpty, e);
          if (old == kEncEmpty || old == e) break;
          h = (h + 1) & (kDedupLdsSlots - 1);
        }
        atomicMin(&lmin[h], static_cast<unsigned int>(i));
        lr[k] = atomicAdd(&lcnt[h], 1u);
        ls[k] = static_cast<int>(h);
      }
    }
  }
  __syncthreads();
  for (int s = tid; s < kDedupLdsSlots; s += kBlock) {
    const unsigned long long e = lkey[s];
    if (e == kEncEmpty) continue;
    uint64_t h = scratch_hash(e) & sc.mask;
    int gs = -1;
    for (uint64_t probe = 0; probe <= sc.mask; ++probe) {
      const unsigned long long old = atomicCAS(&sc.key[h], kEncEmpty, e);
      if (old == kEncEmpty || old == e) {
        gs = static_cast<int>(h);
        break;
      }
      h = (h + 1) & sc.mask;
    }
    if (gs < 0) {
      atomicOr(err, kErrScratch);
      lgs[s] = -1;
      lbase[s] = 0;
      continue;
    }
    atomicMin(&sc.first[gs], lmin[s]);
    lbase[s] = atomicAdd(&sc.cnt[gs], lcnt[s]);
    lgs[s] = gs;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) {
    const int64_t i = base + k * kBlock + tid;
    if (i < n) {
      const int g = ls[k] >= 0 ? lgs[ls[k]] : -1;
      slot_of[i] = g;
      occ_rank[i] = g >= 0 ? static_cast<int>(lbase[ls[k]] + lr[k]) : 0;
    }
  }
}

// Pass 2a: number of first occurrences per tile.
__global__ __launch_bounds__(kBlock) void k_flag_count(const int32_t* __restrict__ slot_of,
                                                       const unsigned int* __restrict__ first, int64_t n,
                                                       int32_t* __restrict__ bsum) {
  __shared__ int sh[kBlock / kWave + 1];
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * kScanItems;
  int v[8];
  load8(slot_of, i0, n, v);
  int c = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t i = i0 + k;
    if (i < n && v[k] >= 0 && first[v[k]] == static_cast<unsigned int>(i)) ++c;
  }
  const int t = block_sum<kBlock>(c, sh);
  if (threadIdx.x == 0) bsum[blockIdx.x] = t;
}

enum : int { kScanDedup = 0, kScanSeg = 1, kScanInsert = 2 };

// Exclusive scan of the tile sums by one 1024-thread block; the total goes
// to the call's scalars.  For the insert scan it also reserves the rows:
// new keys get rows [live, live + inserted) and `live` advances.
__global__ __launch_bounds__(1024) void k_scan_small(int32_t* __restrict__ a, int64_t nb_host,
                                                     const int64_t* len_dev, int tile, int mode,
                                                     int64_t* cscal, int64_t* tscal, int32_t* seg) {
  __shared__ int sh[1024 / kWave + 1];
  const int64_t nb = len_dev ? (*len_dev + tile - 1) / tile : nb_host;
  int carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += 1024) {
    const int64_t idx = b0 + threadIdx.x;
    const int v = idx < nb ? a[idx] : 0;
    int tot;
    const int ex = block_excl_scan<1024>(v, sh, tot);
    if (idx < nb) a[idx] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x != 0) return;
  if (mode == kScanDedup) {
    cscal[kCU] = carry;
  } else if (mode == kScanSeg) {
    cscal[kCValid] = carry;
    seg[*len_dev] = carry;
  } else {
    const int64_t live = tscal[kTLive];
    const int64_t lim = min(tscal[kTLimit], tscal[kTRowCap]);
    const int64_t room = lim > live ? lim - live : 0;
    const int64_t ins = carry < room ? carry : room;
    cscal[kCNew] = ins;
    cscal[kCBaseLive] = live;
    tscal[kTLive] = live + ins;
    if (carry > room) atomicOr(reinterpret_cast<int*>(&tscal[kTErr]), kErrFull);
  }
}

// Pass 2b: ranks of first occurrences -> unique ids; writes unique[], the
// scratch slot and occurrence count of every unique, and slot -> unique id.
__global__ __launch_bounds__(kBlock) void k_compact(const int64_t* __restrict__ values,
                                                    const int32_t* __restrict__ slot_of, Scratch sc,
                                                    int64_t n, const int32_t* __restrict__ bprefix,
                                                    int64_t* __restrict__ unique, int32_t* __restrict__ uslot,
                                                    int32_t* __restrict__ ucount) {
  __shared__ int sh[kBlock / kWave + 1];
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * kScanItems;
  int v[8];
  load8(slot_of, i0, n, v);
  bool f[8];
  int c = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t i = i0 + k;
    f[k] = i < n && v[k] >= 0 && sc.first[v[k]] == static_cast<unsigned int>(i);
    c += f[k];
  }
  int tot;
  int uid = bprefix[blockIdx.x] + block_excl_scan<kBlock>(c, sh, tot);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if (!f[k]) continue;
    const int s = v[k];
    unique[uid] = values[i0 + k];
    uslot[uid] = s;
    ucount[uid] = static_cast<int32_t>(sc.cnt[s]);
    sc.uid[s] = uid;
    ++uid;
  }
}

// Pass 3: inverse[i] = unique id of occurrence i (-1 for a rejected key).
__global__ __launch_bounds__(kBlock) void k_inverse(const int32_t* __restrict__ slot_of,
                                                    const int32_t* __restrict__ suid, int64_t n,
                                                    int32_t* __restrict__ inverse) {
  const int64_t i0 = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * 4;
  if (i0 + 4 <= n) {
    const int4 s = *reinterpret_cast<const int4*>(slot_of + i0);
    int4 o;
    o.x = s.x >= 0 ? suid[s.x] : -1;
    o.y = s.y >= 0 ? suid[s.y] : -1;
    o.z = s.z >= 0 ? suid[s.z] : -1;
    o.w = s.w >= 0 ? suid[s.w] : -1;
    *reinterpret_cast<int4*>(inverse + i0) = o;
  } else {
    for (int64_t i = i0; i < n; ++i) {
      const int s = slot_of[i];
      inverse[i] = s >= 0 ? suid[s] : -1;
    }
  }
}

hipError_t launch_dedup(const int64_t* values, int64_t n, const Scratch& sc, const Work& w, int* err,
                        hipEvent_t* ev_local, hipEvent_t* ev_compact, hipStream_t s) {
  if (n <= 0) {
    (void)hipMemsetAsync(w.scal, 0, sizeof(int64_t) * kCScalars, s);
    return hipGetLastError();
  }
  const unsigned nb = grid_for(n, kScanTile, 1ll << 31);
  if (ev_local && ev_local[0]) (void)hipEventRecord(ev_local[0], s);
  k_dedup_local<<<grid_for(n, kDedupTile, 1ll << 31), kBlock, 0, s>>>(values, n, sc, w.slot_of, w.occ_rank, err);
  if (ev_local && ev_local[1]) (void)hipEventRecord(ev_local[1], s);
  k_flag_count<<<nb, kBlock, 0, s>>>(w.slot_of, sc.first, n, w.bsum);
  k_scan_small<<<1, 1024, 0, s>>>(w.bsum, nb, nullptr, kScanTile, kScanDedup, w.scal, nullptr, nullptr);
  if (ev_compact && ev_compact[0]) (void)hipEventRecord(ev_compact[0], s);
  k_compact<<<nb, kBlock, 0, s>>>(values, w.slot_of, sc, n, w.bsum, w.unique, w.uslot, w.ucount);
  if (ev_compact && ev_compact[1]) (void)hipEventRecord(ev_compact[1], s);
  k_inverse<<<grid_for(n, kBlock * 4, 1ll << 31), kBlock, 0, s>>>(w.slot_of, sc.uid, n, w.inverse);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// occurrence-list segments: seg = exclusive scan of per-unique counts
// ---------------------------------------------------------------------------

// Tile sums of a device-length int array (length *len).
__global__ __launch_bounds__(kBlock) void k_tile_reduce(const int32_t* __restrict__ in, const int64_t* len,
                                                        int32_t* __restrict__ bsum) {
  __shared__ int sh[kBlock / kWave + 1];
  const int64_t L = *len;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
  if (base >= L) return;
  int v[8];
  load8(in, base + threadIdx.x * kScanItems, L, v);
  int c = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) c += v[k];
  const int t = block_sum<kBlock>(c, sh);
  if (threadIdx.x == 0) bsum[blockIdx.x] = t;
}

// seg[u] = occurrences of unique ids < u.  Also returns the dedup scratch
// slots used by this call to empty (so the scratch never needs a full clear),
// and zeroes the partial-sum row of every segment that crosses a chunk
// boundary (its owner chunk is the one holding its first position).
__global__ __launch_bounds__(kBlock) void k_seg_apply(const int32_t* __restrict__ ucount, const int64_t* len,
                                                      const int32_t* __restrict__ bprefix, int32_t* __restrict__ seg,
                                                      const int32_t* __restrict__ uslot, Scratch sc,
                                                      float* __restrict__ gpart, int dim) {
  __shared__ int sh[kBlock / kWave + 1];
  const int64_t L = *len;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
  if (base >= L) return;
  const int64_t i0 = base + threadIdx.x * kScanItems;
  int v[8];
  load8(ucount, i0, L, v);
  int c = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) c += v[k];
  int tot;
  int run = bprefix[blockIdx.x] + block_excl_scan<kBlock>(c, sh, tot);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t u = i0 + k;
    if (u >= L) break;
    seg[u] = run;
    const int st = run, en = run + v[k];
    run = en;
    const int s = uslot[u];
    sc.key[s] = kEncEmpty;
    sc.first[s] = 0xFFFFFFFFu;
    sc.cnt[s] = 0u;
    if (en > st && st / kChunk != (en - 1) / kChunk) {
      float4* p = reinterpret_cast<float4*>(gpart + static_cast<int64_t>(st / kChunk) * dim);
      for (int j = 0; j < dim / 4; ++j) p[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

hipError_t launch_seg_scan(const Work& w, int64_t nmax, const Scratch& sc, int dim, hipStream_t s) {
  if (nmax <= 0) return hipSuccess;
  const unsigned nb = grid_for(nmax, kScanTile, 1ll << 31);
  k_tile_reduce<<<nb, kBlock, 0, s>>>(w.ucount, w.scal + kCU, w.bsum);
  k_scan_small<<<1, 1024, 0, s>>>(w.bsum, 0, w.scal + kCU, kScanTile, kScanSeg, w.scal, nullptr, w.seg);
  k_seg_apply<<<nb, kBlock, 0, s>>>(w.ucount, w.scal + kCU, w.bsum, w.seg, w.uslot, sc, w.gpart, dim);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// IDMap: find (read-only probe), then insert the missing keys
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_idmap_probe(TableDev t, const int64_t* __restrict__ unique,
                                                        const int64_t* len, int64_t* __restrict__ rows,
                                                        int32_t* __restrict__ isnew) {
  const int64_t U = *len;
  for (int64_t u = blockIdx.x * (int64_t)kBlock + threadIdx.x; u < U; u += (int64_t)gridDim.x * kBlock) {
    const unsigned long long e = static_cast<unsigned long long>(unique[u]) ^ kSign;
    const int64_t r = idmap_lookup(t, e);
    rows[u] = r;
    isnew[u] = r < 0 ? 1 : 0;
  }
}

// The initial value of element j of a new key's row: 24 bits of the
// (j+1)-th splitmix64 output from state mix(key ^ mix(seed)), mapped
// exactly onto [0, 1), then one fp32 fused multiply-add onto [lo, hi].
__device__ inline float init_value(uint64_t z, int j, float lo, float span) {
  const uint64_t h = mix64(z + static_cast<uint64_t>(j + 1) * 0x9E3779B97F4A7C15ull);
  const float u = static_cast<float>(h >> 40) * 0x1.0p-24f;
  return __builtin_fmaf(u, span, lo);
}

// New keys of a tile get their global rank (first-occurrence order), then
// lane groups of 16 claim IDMap slots and write the initial rows.
__global__ __launch_bounds__(kBlock) void k_idmap_insert(TableDev t, const int64_t* __restrict__ unique,
                                                         const int32_t* __restrict__ isnew,
                                                         const int32_t* __restrict__ bprefix,
                                                         const int64_t* __restrict__ cscal,
                                                         int64_t* __restrict__ rows) {
  __shared__ int sh[kBlock / kWave + 1];
  __shared__ int list_u[kScanTile];
  __shared__ int list_rank[kScanTile];
  const int64_t U = cscal[kCU];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
  if (base >= U) return;
  const int64_t inserted = cscal[kCNew];
  const int64_t live0 = cscal[kCBaseLive];
  const int64_t i0 = base + threadIdx.x * kScanItems;
  int v[8];
  load8(isnew, i0, U, v);
  int c = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) c += v[k];
  int tot;
  const int lpos = block_excl_scan<kBlock>(c, sh, tot);
  int rank = bprefix[blockIdx.x] + lpos;
  int lp = lpos;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if (!v[k]) continue;
    list_u[lp] = static_cast<int>(i0 + k - base);
    list_rank[lp] = rank;
    ++lp;
    ++rank;
  }
  __syncthreads();
  constexpr int G = 16;
  const int lane = threadIdx.x % G, grp = threadIdx.x / G;
  const int chunks = static_cast<int>(t.store.stride / 16);
  const int wbytes = t.dim * (t.row_dtype ? 2 : 4);
  for (int q = grp; q < tot; q += kBlock / G) {
    const int64_t u = base + list_u[q];
    const int64_t rk = list_rank[q];
    if (rk >= inserted) continue;  // no room: stays -1 (error latched by the scan)
    const int64_t row = live0 + rk;
    const int64_t key = unique[u];
    if (lane == 0) {
      const int64_t slot = idmap_claim(t, static_cast<unsigned long long>(key) ^ kSign);
      if (slot >= 0) {
        t.slots[slot].row = row;
        rows[u] = row;
      } else {
        atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
      }
    }
    const uint64_t z = mix64(static_cast<uint64_t>(key) ^ mix64(t.seed));
    uint8_t* rp = t.store.row(row);
    for (int ch = lane; ch < chunks; ch += G) {
      const int off = ch * 16;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (off < wbytes) {
        if (t.row_dtype == 0) {
          const int j0 = off / 4;
          float f[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) f[k] = init_value(z, j0 + k, t.lo, t.span);
          val = make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
        } else {
          const int j0 = off / 2;
          uint32_t h[4];
#pragma unroll
          for (int k = 0; k < 4; ++k)
            h[k] = static_cast<uint32_t>(f32_to_bf16(init_value(z, j0 + 2 * k, t.lo, t.span))) |
                   (static_cast<uint32_t>(f32_to_bf16(init_value(z, j0 + 2 * k + 1, t.lo, t.span))) << 16);
          val = make_uint4(h[0], h[1], h[2], h[3]);
        }
      }
      *reinterpret_cast<uint4*>(rp + off) = val;
    }
  }
}

hipError_t launch_idmap_probe(const TableDev& t, const Work& w, int64_t nmax, hipEvent_t* ev, hipStream_t s) {
  if (nmax <= 0) return hipSuccess;
  if (ev && ev[0]) (void)hipEventRecord(ev[0], s);
  k_idmap_probe<<<grid_for(nmax, kBlock, 16384), kBlock, 0, s>>>(t, w.unique, w.scal + kCU, w.rows, w.isnew);
  if (ev && ev[1]) (void)hipEventRecord(ev[1], s);
  return hipGetLastError();
}

hipError_t launch_idmap_insert(const TableDev& t, const Work& w, int64_t nmax, hipEvent_t* ev, hipStream_t s) {
  if (nmax <= 0) return hipSuccess;
  const unsigned nb = grid_for(nmax, kScanTile, 1ll << 31);
  k_tile_reduce<<<nb, kBlock, 0, s>>>(w.isnew, w.scal + kCU, w.bsum);
  k_scan_small<<<1, 1024, 0, s>>>(w.bsum, 0, w.scal + kCU, kScanTile, kScanInsert, w.scal, t.scal, nullptr);
  if (ev && ev[0]) (void)hipEventRecord(ev[0], s);
  k_idmap_insert<<<nb, kBlock, 0, s>>>(t, w.unique, w.isnew, w.bsum, w.scal, w.rows);
  if (ev && ev[1]) (void)hipEventRecord(ev[1], s);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_map_rows(const int32_t* __restrict__ inverse,
                                                     const int64_t* __restrict__ rows, int64_t n,
                                                     int64_t* __restrict__ out, const int64_t* cscal,
                                                     int64_t* n_inserted) {
  const int64_t i = blockIdx.x * (int64_t)kBlock + threadIdx.x;
  if (i == 0 && n_inserted) *n_inserted = cscal[kCNew];
  if (i < n) {
    const int u = inverse[i];
    out[i] = u >= 0 ? rows[u] : -1;
  }
}

hipError_t launch_map_rows(const Work& w, int64_t n, int64_t* rows_out, int64_t* n_inserted, hipStream_t s) {
  k_map_rows<<<grid_for(n, kBlock, 1ll << 31), kBlock, 0, s>>>(w.inverse, w.rows, n, rows_out, w.scal, n_inserted);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_find(TableDev t, const int64_t* __restrict__ keys, int64_t n,
                                                 int64_t* __restrict__ out) {
  for (int64_t i = blockIdx.x * (int64_t)kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) {
    const unsigned long long e = static_cast<unsigned long long>(keys[i]) ^ kSign;
    out[i] = e <= kEncTomb ? -1 : idmap_lookup(t, e);
  }
}

hipError_t launch_find(const TableDev& t, const int64_t* keys, int64_t n, int64_t* rows_out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_find<<<grid_for(n, kBlock, 16384), kBlock, 0, s>>>(t, keys, n, rows_out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// forward: fused gather + pool, and the occurrence list for the backward
// ---------------------------------------------------------------------------

// Place occurrence i (of unique u) at its position in u's segment of the
// occurrence list; `ref` is the gradient row it will read in the backward.
__device__ inline void place_occurrence(const Work& w, int u, int64_t i, int ref) {
  const int p = w.seg[u] + w.occ_rank[i];
  w.occ_ref[p] = ref;
  if ((p & (kChunk - 1)) == 0) w.chunk_u[p / kChunk] = u;
}

template <typename WT, int LANES, int MODE>
__global__ __launch_bounds__(kBlock) void k_pool(TableDev t, Work w, const int64_t* __restrict__ offsets,
                                                 int64_t n, int64_t bags, float* __restrict__ out) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  constexpr int D = LANES * E;
  constexpr int GPB = kBlock / LANES;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  for (int64_t g = static_cast<int64_t>(blockIdx.x) * GPB + grp; g < bags; g += static_cast<int64_t>(gridDim.x) * GPB) {
    // CSR bounds clamped to [0, n]: malformed offsets cannot read out of range
    const int64_t b = min(max(offsets[g], int64_t(0)), n);
    const int64_t e = min(max(offsets[g + 1], b), n);
    float acc[E];
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] = 0.f;
    int64_t i = b;
    for (; i + 4 <= e; i += 4) {
      int u[4];
      int64_t r[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) u[q] = w.inverse[i + q];
#pragma unroll
      for (int q = 0; q < 4; ++q) r[q] = u[q] >= 0 ? w.rows[u[q]] : -1;
      float x[4][E];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (r[q] >= 0) {
          load_vals<WT, E>(reinterpret_cast<const WT*>(t.store.row(r[q])) + lane * E, x[q]);
        } else {
#pragma unroll
          for (int k = 0; k < E; ++k) x[q][k] = 0.f;
        }
      }
      if (lane == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (u[q] >= 0) place_occurrence(w, u[q], i + q, static_cast<int>(g));
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < E; ++k) acc[k] += x[q][k];
    }
    for (; i < e; ++i) {
      const int u = w.inverse[i];
      if (u < 0) continue;
      const int64_t r = w.rows[u];
      if (lane == 0) place_occurrence(w, u, i, static_cast<int>(g));
      if (r < 0) continue;
      float x[E];
      load_vals<WT, E>(reinterpret_cast<const WT*>(t.store.row(r)) + lane * E, x);
#pragma unroll
      for (int k = 0; k < E; ++k) acc[k] += x[k];
    }
    if (MODE == 1 && e > b) {
      const float len = static_cast<float>(e - b);
#pragma unroll
      for (int k = 0; k < E; ++k) acc[k] = acc[k] / len;
    }
    store_vals<float, E>(out + g * D + lane * E, acc);
  }
}

template <typename WT, int LANES>
__global__ __launch_bounds__(kBlock) void k_pool_none(TableDev t, Work w, const int64_t* __restrict__ offsets,
                                                      int64_t n, int64_t bags, int64_t L, WT* __restrict__ out,
                                                      uint8_t* __restrict__ mask) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  constexpr int D = LANES * E;
  constexpr int GPB = kBlock / LANES;
  constexpr int TCH = 64;  // positions per block
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t nch = (L + TCH - 1) / TCH;
  for (int64_t blk = blockIdx.x; blk < bags * nch; blk += gridDim.x) {
    const int64_t g = blk / nch, c = blk % nch;
    const int64_t b = min(max(offsets[g], int64_t(0)), n);
    const int64_t len = min(max(offsets[g + 1], b), n) - b;
    for (int tt = grp; tt < TCH; tt += GPB) {
      const int64_t tpos = c * TCH + tt;
      if (tpos >= L) break;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (tpos < len) {
        const int u = w.inverse[b + tpos];
        const int64_t r = u >= 0 ? w.rows[u] : -1;
        if (r >= 0) v = *reinterpret_cast<const uint4*>(reinterpret_cast<const WT*>(t.store.row(r)) + lane * E);
        if (lane == 0 && u >= 0) place_occurrence(w, u, b + tpos, static_cast<int>(g * L + tpos));
      }
      *reinterpret_cast<uint4*>(out + (g * L + tpos) * D + lane * E) = v;
      if (lane == 0) mask[g * L + tpos] = tpos < len ? 1 : 0;
    }
    if (c == 0 && lane == 0) {
      // ids past pad_len: in the occurrence list (the key is touched) but
      // without a gradient row
      for (int64_t tpos = L + grp; tpos < len; tpos += GPB) {
        const int u = w.inverse[b + tpos];
        if (u >= 0) place_occurrence(w, u, b + tpos, -1);
      }
    }
  }
}

template <typename WT, int LANES>
static hipError_t pool_dispatch_mode(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags,
                                     int mode, int64_t pad_len, void* out, uint8_t* mask, hipStream_t s) {
  constexpr int GPB = kBlock / LANES;
  if (mode == 2) {
    const int64_t nch = (pad_len + 63) / 64;
    k_pool_none<WT, LANES><<<grid_for(bags * nch, 1, 1 << 20), kBlock, 0, s>>>(
        t, w, offsets, n, bags, pad_len, static_cast<WT*>(out), mask);
  } else if (mode == 1) {
    k_pool<WT, LANES, 1><<<grid_for(bags, GPB, 1 << 20), kBlock, 0, s>>>(t, w, offsets, n, bags, static_cast<float*>(out));
  } else {
    k_pool<WT, LANES, 0><<<grid_for(bags, GPB, 1 << 20), kBlock, 0, s>>>(t, w, offsets, n, bags, static_cast<float*>(out));
  }
  return hipGetLastError();
}

template <typename WT>
static hipError_t pool_dispatch_dim(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags,
                                    int mode, int64_t pad_len, void* out, uint8_t* mask, hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(WT));
  switch (t.dim / E) {
    case 1: return pool_dispatch_mode<WT, 1>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 2: return pool_dispatch_mode<WT, 2>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 4: return pool_dispatch_mode<WT, 4>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 8: return pool_dispatch_mode<WT, 8>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 16: return pool_dispatch_mode<WT, 16>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 32: return pool_dispatch_mode<WT, 32>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    case 64: return pool_dispatch_mode<WT, 64>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_pool(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags, int mode,
                       int64_t pad_len, void* out, uint8_t* mask, hipEvent_t* ev, hipStream_t s) {
  if (bags <= 0) return hipSuccess;
  if (ev && ev[0]) (void)hipEventRecord(ev[0], s);
  hipError_t e = t.row_dtype ? pool_dispatch_dim<uint16_t>(t, w, offsets, n, bags, mode, pad_len, out, mask, s)
                             : pool_dispatch_dim<float>(t, w, offsets, n, bags, mode, pad_len, out, mask, s);
  if (ev && ev[1]) (void)hipEventRecord(ev[1], s);
  return e;
}

// ---------------------------------------------------------------------------
// backward: per-unique gradient sums over the occurrence list, fused with
// the optimizer update of the row
// ---------------------------------------------------------------------------

// Row-sparse optimizer on E consecutive elements [lane*E, lane*E + E) of a row.
template <typename WT, int E>
__device__ inline void apply_opt(uint8_t* row, int lane, int dim, const float (&g)[E], const OptArgs& o) {
  WT* wp = reinterpret_cast<WT*>(row) + lane * E;
  float* s1 = reinterpret_cast<float*>(row + static_cast<int64_t>(dim) * sizeof(WT)) + lane * E;
  float w[E], a[E];
  load_vals<WT, E>(wp, w);
  load_vals<float, E>(s1, a);
  if (o.opt == 0) {
#pragma unroll
    for (int k = 0; k < E; ++k) {
      a[k] = a[k] + g[k] * g[k];
      w[k] = w[k] - o.lr * g[k] / (__builtin_sqrtf(a[k]) + o.eps);
    }
    store_vals<float, E>(s1, a);
  } else {
    float* s2 = s1 + dim;
    float v[E];
    load_vals<float, E>(s2, v);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      a[k] = o.beta1 * a[k] + o.omb1 * g[k];
      v[k] = o.beta2 * v[k] + o.omb2 * g[k] * g[k];
      w[k] = w[k] - o.lr * (a[k] / o.bc1) / (__builtin_sqrtf(v[k] / o.bc2) + o.eps);
    }
    store_vals<float, E>(s1, a);
    store_vals<float, E>(s2, v);
  }
  store_vals<WT, E>(wp, w);
}

template <typename WT, int E, bool FUSED>
__device__ inline void finish_unique(const TableDev& t, const Work& w, int u, int lane, const float (&acc)[E],
                                     float* grad_unique, const OptArgs& o) {
  if (FUSED) {
    const int64_t r = w.rows[u];
    if (r >= 0) apply_opt<WT, E>(t.store.row(r), lane, t.dim, acc, o);
  } else {
    store_vals<float, E>(grad_unique + static_cast<int64_t>(u) * t.dim + lane * E, acc);
  }
}

// Gradient of one occurrence-list position: scale * grad row `ref`.
template <typename GT, int E, int MODE>
__device__ inline void add_grad(const GT* __restrict__ grad, const int64_t* __restrict__ offsets, int ref,
                                int lane, int dim, float (&acc)[E]) {
  float x[E];
  load_vals<GT, E>(grad + static_cast<int64_t>(ref) * dim + lane * E, x);
  if (MODE == 1) {
    const float sc = 1.0f / static_cast<float>(offsets[ref + 1] - offsets[ref]);
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] += sc * x[k];
  } else {
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] += x[k];
  }
}

// One lane group per chunk of kChunk consecutive occurrence-list positions.
// A segment (all positions of one unique id) lying inside the chunk is
// finished here; a segment crossing a chunk boundary has its partial sum
// added into the partial row of its owner chunk and is finished by
// k_bwd_straddle.
template <typename WT, typename GT, int LANES, int MODE, bool FUSED>
__global__ __launch_bounds__(kBlock) void k_bwd_chunks(TableDev t, Work w, const int64_t* __restrict__ offsets,
                                                       const GT* __restrict__ grad, float* __restrict__ grad_unique,
                                                       OptArgs o) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  constexpr int GPB = kBlock / LANES;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int dim = LANES * E;
  const int64_t total = w.scal[kCValid];
  const int64_t nch = (total + kChunk - 1) / kChunk;
  for (int64_t c = static_cast<int64_t>(blockIdx.x) * GPB + grp; c < nch; c += static_cast<int64_t>(gridDim.x) * GPB) {
    const int64_t p0 = c * kChunk;
    const int64_t p1 = min(p0 + kChunk, total);
    int u = w.chunk_u[c];
    while (true) {
      const int64_t s = w.seg[u], e = w.seg[u + 1];
      const int64_t pa = max(s, p0), pb = min(e, p1);
      float acc[E];
#pragma unroll
      for (int k = 0; k < E; ++k) acc[k] = 0.f;
      int64_t p = pa;
      for (; p + 4 <= pb; p += 4) {
        int ref[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) ref[q] = w.occ_ref[p + q];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (ref[q] >= 0) add_grad<GT, E, MODE>(grad, offsets, ref[q], lane, dim, acc);
      }
      for (; p < pb; ++p) {
        const int ref = w.occ_ref[p];
        if (ref >= 0) add_grad<GT, E, MODE>(grad, offsets, ref, lane, dim, acc);
      }
      if (s >= p0 && e <= p1) {
        finish_unique<WT, E, FUSED>(t, w, u, lane, acc, grad_unique, o);
      } else {
        float* gp = w.gpart + (s / kChunk) * dim + lane * E;
#pragma unroll
        for (int k = 0; k < E; ++k) unsafeAtomicAdd(gp + k, acc[k]);
      }
      if (e >= p1) break;
      ++u;
    }
  }
}

template <typename WT, int LANES, int E, bool FUSED>
__global__ __launch_bounds__(kBlock) void k_bwd_straddle(TableDev t, Work w, float* __restrict__ grad_unique,
                                                         OptArgs o) {
  constexpr int GPB = kBlock / LANES;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int dim = LANES * E;
  const int64_t U = w.scal[kCU];
  for (int64_t u = static_cast<int64_t>(blockIdx.x) * GPB + grp; u < U; u += static_cast<int64_t>(gridDim.x) * GPB) {
    const int s = w.seg[u], e = w.seg[u + 1];
    if (e <= s || s / kChunk == (e - 1) / kChunk) continue;
    float acc[E];
    load_vals<float, E>(w.gpart + static_cast<int64_t>(s / kChunk) * dim + lane * E, acc);
    finish_unique<WT, E, FUSED>(t, w, static_cast<int>(u), lane, acc, grad_unique, o);
  }
}

template <typename WT, typename GT, int LANES, int MODE, bool FUSED>
static hipError_t bwd_launch(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, const void* grad,
                             float* grad_unique, const OptArgs& o, hipEvent_t* ev_c, hipEvent_t* ev_s,
                             hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  constexpr int GPB = kBlock / LANES;
  const int64_t nch_max = (n + kChunk - 1) / kChunk;
  if (ev_c && ev_c[0]) (void)hipEventRecord(ev_c[0], s);
  k_bwd_chunks<WT, GT, LANES, MODE, FUSED><<<grid_for(nch_max, GPB, 1 << 20), kBlock, 0, s>>>(
      t, w, offsets, static_cast<const GT*>(grad), grad_unique, o);
  if (ev_c && ev_c[1]) (void)hipEventRecord(ev_c[1], s);
  if (ev_s && ev_s[0]) (void)hipEventRecord(ev_s[0], s);
  k_bwd_straddle<WT, LANES, E, FUSED><<<grid_for(n, GPB, 1 << 16), kBlock, 0, s>>>(t, w, grad_unique, o);
  if (ev_s && ev_s[1]) (void)hipEventRecord(ev_s[1], s);
  return hipGetLastError();
}

template <typename WT, typename GT, int MODE, bool FUSED>
static hipError_t bwd_dim(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, const void* grad,
                          float* gu, const OptArgs& o, hipEvent_t* ec, hipEvent_t* es, hipStream_t s) {
  constexpr int E = 16 / static_cast<int>(sizeof(GT));
  switch (t.dim / E) {
    case 1: return bwd_launch<WT, GT, 1, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 2: return bwd_launch<WT, GT, 2, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 4: return bwd_launch<WT, GT, 4, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 8: return bwd_launch<WT, GT, 8, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 16: return bwd_launch<WT, GT, 16, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 32: return bwd_launch<WT, GT, 32, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    case 64: return bwd_launch<WT, GT, 64, MODE, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename WT, bool FUSED>
static hipError_t bwd_mode(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int mode,
                           const void* grad, float* gu, const OptArgs& o, hipEvent_t* ec, hipEvent_t* es,
                           hipStream_t s) {
  if (mode == 2) return bwd_dim<WT, WT, 0, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
  if (mode == 1) return bwd_dim<WT, float, 1, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
  return bwd_dim<WT, float, 0, FUSED>(t, w, offsets, n, grad, gu, o, ec, es, s);
}

hipError_t launch_bwd(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t /*bags*/,
                      int mode, int64_t /*pad_len*/, const void* grad, float* grad_unique, const OptArgs* opt,
                      hipEvent_t* ev_chunks, hipEvent_t* ev_straddle, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const OptArgs o = opt ? *opt : OptArgs{0, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 1.f, 1.f};
  if (opt) {
    return t.row_dtype ? bwd_mode<uint16_t, true>(t, w, offsets, n, mode, grad, grad_unique, o, ev_chunks, ev_straddle, s)
                       : bwd_mode<float, true>(t, w, offsets, n, mode, grad, grad_unique, o, ev_chunks, ev_straddle, s);
  }
  return t.row_dtype ? bwd_mode<uint16_t, false>(t, w, offsets, n, mode, grad, grad_unique, o, ev_chunks, ev_straddle, s)
                     : bwd_mode<float, false>(t, w, offsets, n, mode, grad, grad_unique, o, ev_chunks, ev_straddle, s);
}

// ---------------------------------------------------------------------------
// optimizer from a written grad_unique
// ---------------------------------------------------------------------------

template <typename WT, int LANES>
__global__ __launch_bounds__(kBlock) void k_opt(TableDev t, Work w, const float* __restrict__ grad_unique, OptArgs o) {
  constexpr int E = 4;
  constexpr int GPB = kBlock / LANES;
  const int lane = threadIdx.x % LANES;
  const int grp = threadIdx.x / LANES;
  const int64_t U = w.scal[kCU];
  for (int64_t u = static_cast<int64_t>(blockIdx.x) * GPB + grp; u < U; u += static_cast<int64_t>(gridDim.x) * GPB) {
    const int64_t r = w.rows[u];
    if (r < 0) continue;
    float g[E];
    load_vals<float, E>(grad_unique + u * t.dim + lane * E, g);
    apply_opt<WT, E>(t.store.row(r), lane, t.dim, g, o);
  }
}

template <typename WT>
static hipError_t opt_dim(const TableDev& t, const Work& w, int64_t n, const float* gu, const OptArgs& o, hipStream_t s) {
  switch (t.dim / 4) {
    case 2: k_opt<WT, 2><<<grid_for(n, kBlock / 2, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    case 4: k_opt<WT, 4><<<grid_for(n, kBlock / 4, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    case 8: k_opt<WT, 8><<<grid_for(n, kBlock / 8, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    case 16: k_opt<WT, 16><<<grid_for(n, kBlock / 16, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    case 32: k_opt<WT, 32><<<grid_for(n, kBlock / 32, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    case 64: k_opt<WT, 64><<<grid_for(n, kBlock / 64, 1 << 16), kBlock, 0, s>>>(t, w, gu, o); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_opt(const TableDev& t, const Work& w, int64_t n, const float* grad_unique, const OptArgs& opt,
                      hipEvent_t* ev, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (ev && ev[0]) (void)hipEventRecord(ev[0], s);
  hipError_t e = t.row_dtype ? opt_dim<uint16_t>(t, w, n, grad_unique, opt, s) : opt_dim<float>(t, w, n, grad_unique, opt, s);
  if (ev && ev[1]) (void)hipEventRecord(ev[1], s);
  return e;
}

// ---------------------------------------------------------------------------
// table maintenance: rehash, export, read rows
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_rehash(const Slot* __restrict__ old, int64_t old_cap, TableDev t) {
  for (int64_t i = blockIdx.x * (int64_t)kBlock + threadIdx.x; i < old_cap; i += (int64_t)gridDim.x * kBlock) {
    const Slot sl = old[i];
    if (sl.key <= kEncTomb) continue;
    const int64_t slot = idmap_claim(t, sl.key);
    if (slot >= 0) t.slots[slot].row = sl.row;
    else atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
  }
}

hipError_t launch_rehash(const Slot* old_slots, int64_t old_cap, const TableDev& t, hipStream_t s) {
  k_rehash<<<grid_for(old_cap, kBlock, 65536), kBlock, 0, s>>>(old_slots, old_cap, t);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_export(TableDev t, int64_t cap_slots, int64_t* __restrict__ keys,
                                                   int64_t* __restrict__ rows, int64_t cap, unsigned long long* counter) {
  for (int64_t i = blockIdx.x * (int64_t)kBlock + threadIdx.x; i < cap_slots; i += (int64_t)gridDim.x * kBlock) {
    const Slot sl = t.slots[i];
    if (sl.key <= kEncTomb) continue;
    const unsigned long long k = atomicAdd(counter, 1ull);
    if (static_cast<int64_t>(k) < cap) {
      keys[k] = static_cast<int64_t>(sl.key ^ kSign);
      rows[k] = sl.row;
    }
  }
}

__global__ void k_copy_scalar(const int64_t* src, int64_t* dst) { *dst = *src; }

hipError_t launch_export(const TableDev& t, int64_t cap_slots, int64_t* keys, int64_t* rows, int64_t cap,
                         int64_t* n_dev, hipStream_t s) {
  (void)hipMemsetAsync(&t.scal[kTExport], 0, sizeof(int64_t), s);
  k_export<<<grid_for(cap_slots, kBlock, 65536), kBlock, 0, s>>>(
      t, cap_slots, keys, rows, cap, reinterpret_cast<unsigned long long*>(&t.scal[kTExport]));
  if (n_dev) k_copy_scalar<<<1, 1, 0, s>>>(&t.scal[kTExport], n_dev);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_read_rows(TableDev t, const int64_t* __restrict__ rows, int64_t n,
                                                      float* __restrict__ w_out, float* __restrict__ state_out) {
  const int64_t live = t.scal[kTLive];
  const int64_t total = n * t.dim;
  for (int64_t idx = blockIdx.x * (int64_t)kBlock + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * kBlock) {
    const int64_t i = idx / t.dim;
    const int j = static_cast<int>(idx % t.dim);
    const int64_t r = rows[i];
    const bool ok = r >= 0 && r < live;
    const uint8_t* rp = ok ? t.store.row(r) : nullptr;
    if (w_out) {
      float v = __builtin_nanf("");
      if (ok) v = t.row_dtype ? bf16_to_f32(reinterpret_cast<const uint16_t*>(rp)[j]) : reinterpret_cast<const float*>(rp)[j];
      w_out[idx] = v;
    }
    if (state_out) {
      const float* sp = ok ? reinterpret_cast<const float*>(rp + static_cast<int64_t>(t.dim) * (t.row_dtype ? 2 : 4)) : nullptr;
      for (int q = 0; q < t.nstate; ++q)
        state_out[(i * t.nstate + q) * t.dim + j] = ok ? sp[q * t.dim + j] : __builtin_nanf("");
    }
  }
}

hipError_t launch_read_rows(const TableDev& t, const int64_t* rows, int64_t n, float* w_out, float* state_out,
                            hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_read_rows<<<grid_for(n * t.dim, kBlock, 65536), kBlock, 0, s>>>(t, rows, n, w_out, state_out);
  return hipGetLastError();
}

}  // namespace rs

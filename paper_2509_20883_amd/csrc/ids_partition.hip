// Ids partition (gfx950): dedup of a batch of ids fused with the split of the
// distinct ids by the shard that owns them (RecIS, "Ids Partition" among the
// benchmarked operators; "Request Merging & Sharding": requests are
// deduplicated and sharded by id before the all-to-all).
//
// owner(k) = mix64(uint64(k) ^ seed) mod G.  Output: the distinct keys shard
// by shard, each shard's keys in first-occurrence order, the shard offsets,
// and each id's position in that list.
//
// Passes (the first two are the lookup's dedup passes with no IDMap):
//   k_tile_dedup, k_part_dedup   key index, first position and count of
//                                every distinct key; its first record flagged
//                                (records are in first-position order)
//   k_owner_hist     per block of record slots: distinct keys (first
//                    records) per owner, in LDS
//   k_scan_one / k_scan_flat  exclusive scan of those counts in (shard,
//                    block) order (one block, or chunks + a last-block pass)
//   k_owner_scatter  per block, in record order: stable rank of each first
//                    record among its shard's (wave ballots on the owner
//                    bits), key to its output slot, slot by key index
//   k_ids_inverse    per id: the output slot of its key (id -> record -> key
//                    index -> slot)
#include "device_common.h"

#include <algorithm>

namespace rs {

__device__ inline uint32_t owner_of(int64_t key, uint64_t seed, uint32_t G, uint32_t gmask) {
  const uint64_t h = mix64(static_cast<uint64_t>(key) ^ seed);
  // G a power of two: the mask is the same residue
  return gmask ? static_cast<uint32_t>(h & gmask) : static_cast<uint32_t>(h % G);
}

OwnerGeom owner_geom(int64_t n, int G) {
  OwnerGeom og;
  const int64_t n1 = n > 0 ? n : 1;
  // rank tiles per block: as few as keep the count table (G per block) at
  // most a quarter of the ids (or 16384 counts) and within one two-level scan
  const int64_t cap = std::min<int64_t>(std::max<int64_t>(n1 / 4, 16384), int64_t(kScanChunk) * kScanChunk);
  og.ch = 1;
  og.nb = (n1 + kRankTile - 1) / kRankTile;
  while (static_cast<int64_t>(G) * og.nb > cap) {
    og.ch <<= 1;
    og.nb = (n1 + og.ch * kRankTile - 1) / (og.ch * kRankTile);
  }
  og.len = static_cast<int64_t>(G) * og.nb;
  og.nch = (og.len + kScanChunk - 1) / kScanChunk;
  og.nbits = 0;
  while ((1 << og.nbits) < G) ++og.nbits;
  og.gmask = (G & (G - 1)) == 0 ? static_cast<uint32_t>(G - 1) : 0u;
  return og;
}

// The owner passes walk the dedup records, whose record tiles (block-major,
// kRankTile record slots each) list every key once, at its first record, in
// the order of the keys' first positions.  "Position" b below is a record
// slot: record tile b / kRankTile, slot b % kRankTile; item k of thread t is
// slot k * kBlock + t (item-major, then thread: ascending record order).
// f[k]: the key index of a first record, else -1; v[k]: its key (from the
// partition-ordered copy, whose entry at the key index is that record).
__device__ inline void load_tile(const Work& w, int64_t b, int (&f)[kRankItems], int64_t (&v)[kRankItems]) {
  const int64_t per = w.g.rcap / kRankTile;
  const int64_t rt = b / kRankTile;
  const int64_t blk = rt / per;
  const int64_t base = blk * w.g.rcap + (rt % per) * kRankTile;
  const int64_t nr = blk * w.g.rcap + w.nrec[blk];
  int2 r[kRankItems];
#pragma unroll
  for (int k = 0; k < kRankItems; ++k) r[k] = w.recres[base + k * kBlock + threadIdx.x];
#pragma unroll
  for (int k = 0; k < kRankItems; ++k) {
    const int64_t j = base + k * kBlock + threadIdx.x;
    f[k] = j < nr && (static_cast<uint32_t>(r[k].y) & kRecFirst) ? r[k].x : -1;
  }
#pragma unroll
  for (int k = 0; k < kRankItems; ++k)
    v[k] = f[k] >= 0 ? static_cast<int64_t>(w.srec[f[k]].key ^ kSign) : 0;  // all in flight together
}

__global__ __launch_bounds__(kBlock) void k_owner_hist(Work w, int64_t n, int G, uint64_t seed, OwnerGeom og,
                                                       int32_t* __restrict__ hist) {
  __shared__ int lh[kMaxShards];
  for (int q = threadIdx.x; q < G; q += kBlock) lh[q] = 0;
  __syncthreads();
  const int64_t base = static_cast<int64_t>(blockIdx.x) * og.ch * kRankTile;
  for (int64_t c = 0; c < og.ch; ++c) {
    const int64_t b = base + c * kRankTile;
    if (b >= n) break;  // block-uniform
    int f[kRankItems];
    int64_t v[kRankItems];
    load_tile(w, b, f, v);
#pragma unroll
    for (int k = 0; k < kRankItems; ++k)
      if (f[k] >= 0) atomicAdd(&lh[owner_of(v[k], seed, G, og.gmask)], 1);
  }
  __syncthreads();
  for (int q = threadIdx.x; q < G; q += kBlock) hist[static_cast<int64_t>(q) * og.nb + blockIdx.x] = lh[q];
}

// In-place exclusive scan of a[0, len): block c scans chunk c and stores its
// total; the last block to finish (a counter, no waiting) scans the chunk
// totals (nch <= kScanChunk).  An element's prefix is then
// a[j] + csum[j / kScanChunk]; the grand total goes to *total.
template <int R>
__global__ __launch_bounds__(1024) void k_scan_flat(int32_t* __restrict__ a, int64_t len, int32_t* __restrict__ csum,
                                                    int64_t nch, int64_t* counter, int64_t* total) {
  static_assert(1024 * R == kScanChunk, "one chunk per block");
  __shared__ int sh[1024 / kWave + 1];
  __shared__ bool last;
  const int64_t c = blockIdx.x;
  const int64_t lo = c * kScanChunk + static_cast<int64_t>(threadIdx.x) * R;
  int v[R];
  int loc = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    v[j] = lo + j < len ? a[lo + j] : 0;
    loc += v[j];
  }
  int tot;
  int run = block_excl_scan<1024>(loc, sh, tot);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if (lo + j < len) a[lo + j] = run;
    run += v[j];
  }
  if (nch == 1) {
    if (threadIdx.x == 0) {
      csum[0] = 0;
      *total = tot;
    }
    return;
  }
  if (threadIdx.x == 0) {
    csum[c] = tot;
    __threadfence();
    const unsigned long long done = atomicAdd(reinterpret_cast<unsigned long long*>(counter), 1ull);
    last = done == static_cast<unsigned long long>(nch - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  const int64_t clo = static_cast<int64_t>(threadIdx.x) * R;
  int cv[R];
  loc = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    cv[j] = clo + j < nch ? __hip_atomic_load(&csum[clo + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    loc += cv[j];
  }
  run = block_excl_scan<1024>(loc, sh, tot);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if (clo + j < nch) csum[clo + j] = run;
    run += cv[j];
  }
  if (threadIdx.x == 0) {
    *counter = 0;  // ready for the next call on this workspace
    *total = tot;
  }
}

// One-block exclusive scan of a[0, len), len <= 1024 R, in place; the chunk
// offsets csum[0, nch) are all zero, so prefixes read as in k_scan_flat.
// Wave w owns elements [64 R w, 64 R (w + 1)): its j-th row of 64 is one
// coalesced load, scanned across the lanes and chained over the rows.
template <int R>
__global__ __launch_bounds__(1024) void k_scan_one(int32_t* __restrict__ a, int64_t len, int32_t* __restrict__ csum,
                                                   int64_t nch, int64_t* total) {
  constexpr int NW = 1024 / kWave;
  __shared__ int sh[NW + 1];
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  const int64_t base = static_cast<int64_t>(wid) * R * kWave + lane;
  int v[R];
#pragma unroll
  for (int j = 0; j < R; ++j) v[j] = base + j * kWave < len ? a[base + j * kWave] : 0;
  int ex[R];
  int run = 0;  // the wave's total over rows < j
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int inc = wave_incl_scan(v[j]);
    ex[j] = run + inc - v[j];
    run += __shfl(inc, kWave - 1, kWave);
  }
  if (lane == 0) sh[wid] = run;
  __syncthreads();
  if (wid == 0) {  // one wave scans the per-wave totals
    const int t = lane < NW ? sh[lane] : 0;
    const int i2 = wave_incl_scan(t);
    if (lane < NW) sh[lane] = i2 - t;
    if (lane == kWave - 1) sh[NW] = i2;
  }
  __syncthreads();
  const int off = sh[wid];
#pragma unroll
  for (int j = 0; j < R; ++j)
    if (base + j * kWave < len) a[base + j * kWave] = off + ex[j];
  if (threadIdx.x < nch) csum[threadIdx.x] = 0;
  if (threadIdx.x == 0) *total = sh[NW];
}

__global__ __launch_bounds__(kBlock) void k_owner_scatter(Work w, int64_t n, int G,
                                                          uint64_t seed, OwnerGeom og, const int32_t* __restrict__ hist,
                                                          const int32_t* __restrict__ csum,
                                                          int32_t* __restrict__ kslot, const int64_t* pscal,
                                                          int64_t* __restrict__ keys_out,
                                                          int64_t* __restrict__ shard_offsets, int64_t* info) {
  constexpr int NW = kBlock / kWave;
  __shared__ int run[kMaxShards];     // next output slot of each shard
  __shared__ int wc[NW][kMaxShards];  // this round's first occurrences per (wave, shard)
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
  const int64_t blk = blockIdx.x;
  for (int q = tid; q < G; q += kBlock) {
    const int64_t j = static_cast<int64_t>(q) * og.nb + blk;
    const int p = hist[j] + csum[j / kScanChunk];
    run[q] = p;
#pragma unroll
    for (int u = 0; u < NW; ++u) wc[u][q] = 0;
    if (blk == 0) shard_offsets[q] = p;
  }
  if (blk == 0 && tid == 0) {
    const int64_t U = pscal[kPTotal];
    shard_offsets[G] = U;
    info[0] = U;
    info[1] = pscal[kTErr];
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
  const int64_t base = blk * og.ch * kRankTile;
  for (int64_t c = 0; c < og.ch; ++c) {
    const int64_t b = base + c * kRankTile;
    if (b >= n) break;  // block-uniform
    int f[kRankItems];
    int64_t v[kRankItems];
    load_tile(w, b, f, v);
    uint32_t own[kRankItems];
#pragma unroll
    for (int k = 0; k < kRankItems; ++k) own[k] = f[k] >= 0 ? owner_of(v[k], seed, G, og.gmask) : 0u;
    // item k of every thread, in position order: waves 0..NW-1, lanes 0..63
#pragma unroll
    for (int k = 0; k < kRankItems; ++k) {
      const bool valid = f[k] >= 0;
      // lanes of this wave whose first occurrence has the same owner
      uint64_t peers = __ballot(valid);
      for (int bit = 0; bit < og.nbits; ++bit) {
        const bool on = (own[k] >> bit) & 1u;
        const uint64_t bb = __ballot(on);
        peers &= on ? bb : ~bb;
      }
      const int cnt = __popcll(peers);
      const bool leader = valid && (peers & below) == 0ull;
      if (leader) wc[wid][own[k]] = cnt;
      __syncthreads();
      if (valid) {
        int pos = run[own[k]] + __popcll(peers & below);
        for (int u = 0; u < wid; ++u) pos += wc[u][own[k]];
        keys_out[pos] = v[k];
        kslot[f[k]] = pos;
      }
      __syncthreads();
      if (leader) {
        atomicAdd(&run[own[k]], cnt);
        wc[wid][own[k]] = 0;
      }
      __syncthreads();
    }
  }
}

// inverse[i] = output slot of occurrence i's key: its dedup record (from the
// occurrence word), the record's key index, that key's slot; -1 for a
// rejected (reserved) key.
__global__ __launch_bounds__(kBlock) void k_ids_inverse(Work w, const int32_t* __restrict__ kslot, int64_t n) {
  const int64_t i0 = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * 4;
  if (i0 >= n) return;
  const FrontGeom g = w.g;
  uint32_t o[4];
  if (i0 + 4 <= n) {
    const uint4 a = *reinterpret_cast<const uint4*>(w.occ_word + i0);
    o[0] = a.x;
    o[1] = a.y;
    o[2] = a.z;
    o[3] = a.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = i0 + k < n ? w.occ_word[i0 + k] : kOccRejected;
  }
  int kid[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {  // all four record reads in flight together
    const bool rej = o[k] == kOccRejected;
    const int64_t src = rej ? 0 : ((i0 + k) >> kDedupTileLog2) / g.R * g.rcap + (o[k] >> 12);
    const int x = w.recres[src].x;
    kid[k] = rej ? -1 : x;
  }
  int pos[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) pos[k] = kid[k] < 0 ? -1 : kslot[kid[k]];
  if (i0 + 4 <= n) {
    *reinterpret_cast<int4*>(w.inverse + i0) = make_int4(pos[0], pos[1], pos[2], pos[3]);
  } else {
    for (int k = 0; k < 4 && i0 + k < n; ++k) w.inverse[i0 + k] = pos[k];
  }
}

__global__ void k_ids_init(int64_t* pscal, int64_t n, int G, int64_t* shard_offsets, int64_t* info) {
  const int tid = threadIdx.x;
  if (tid < kPScalars) pscal[tid] = 0;
  if (n > 0) return;
  for (int q = tid; q <= G; q += blockDim.x) shard_offsets[q] = 0;
  if (tid == 0) {
    info[0] = 0;
    info[1] = 0;
  }
}

hipError_t launch_ids_partition(const int64_t* values, int64_t n, int G, uint64_t seed, const Work& w,
                                const OwnerGeom& og, int32_t* hist, int32_t* csum, int32_t* kslot, int64_t* pscal,
                                int64_t* keys_out, int64_t* shard_offsets, int64_t* info, hipStream_t s) {
  if (G < 1 || G > kMaxShards || og.nch > kScanChunk) return hipErrorInvalidValue;
  k_ids_init<<<1, kBlock, 0, s>>>(pscal, n, G, shard_offsets, info);
  if (n <= 0) return hipGetLastError();
  // no IDMap: the dedup passes probe nothing; their error bits go to pscal
  TableDev t{};
  t.scal = pscal;
  hipError_t e = launch_dedup_keys(values, n, t, w, nullptr, nullptr, s);
  if (e != hipSuccess) return e;
  // the owner passes walk the record slots of the dedup blocks
  const int64_t nslots = record_tiles(w.g) * kRankTile;
  k_owner_hist<<<static_cast<unsigned>(og.nb), kBlock, 0, s>>>(w, nslots, G, seed, og, hist);
  constexpr int kOneBlock = 16;  // counts per thread of the one-block scan
  if (og.len <= 1024 * kOneBlock)
    k_scan_one<kOneBlock><<<1, 1024, 0, s>>>(hist, og.len, csum, og.nch, pscal + kPTotal);
  else
    k_scan_flat<kScanChunk / 1024><<<static_cast<unsigned>(og.nch), 1024, 0, s>>>(hist, og.len, csum, og.nch,
                                                                                  pscal + kPCounter, pscal + kPTotal);
  k_owner_scatter<<<static_cast<unsigned>(og.nb), kBlock, 0, s>>>(w, nslots, G, seed, og, hist, csum, kslot, pscal,
                                                                  keys_out, shard_offsets, info);
  k_ids_inverse<<<grid_for(n, kBlock * 4, 1ll << 31), kBlock, 0, s>>>(w, kslot, n);
  return hipGetLastError();
}

}  // namespace rs

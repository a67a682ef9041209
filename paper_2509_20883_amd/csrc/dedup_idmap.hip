// Dedup and IDMap kernels of the sparse embedding step (gfx950).
//
// RecIS keeps a two-tier store: an IDMap from feature id to an offset and
// Blocks holding the rows ("Optimization for Memory Bound"); ids are
// deduplicated before the lookup ("ids partition").  One forward runs:
//   k_dedup_local    per 1024-occurrence tile: LDS dedup, then one global
//                    scratch insert per distinct key of the tile (atomicMin of
//                    its first position, atomicAdd of its count; the value the
//                    atomicAdd returns ranks the tile's occurrences of the key)
//   k_rank_probe     first occurrences probe the IDMap; tile sums of
//                    (first occurrences, their counts, keys not found, hot
//                    keys, backward units of the hot keys)
//   k_scan5          one block scans the five tile-sum arrays and reserves
//                    the rows of the new keys
//   k_compact_insert unique ids in first-occurrence order, occurrence-list
//                    segments, rows; new keys claim an IDMap slot
//   k_occ_init       per occurrence: unique id (inverse), row, position in the
//                    occurrence list, hot-key backward units; releases the
//                    scratch slots.  Its other blocks write the initial rows
//                    of the new keys
#include "device_common.h"

namespace rs {

// ---------------------------------------------------------------------------
// open addressing (linear probing)
// ---------------------------------------------------------------------------

// Row of an encoded key, or -1 when the probe reaches an empty slot; the
// probe starts `done` slots into the key's sequence (at slot h).  Reads
// kProbeBatch consecutive slots per round trip.
__device__ inline int64_t idmap_lookup_at(const TableDev& t, unsigned long long e, uint64_t h, uint64_t done) {
  for (uint64_t probed = done; probed <= t.cap_mask; probed += kProbeBatch) {
    Slot sl[kProbeBatch];
#pragma unroll
    for (int k = 0; k < kProbeBatch; ++k) sl[k] = t.slots[(h + k) & t.cap_mask];
    int64_t r = -1;
    bool fin = false;
#pragma unroll
    for (int k = 0; k < kProbeBatch; ++k) {  // selects only: the batch stays in registers
      const bool hit = !fin && sl[k].key == e;
      const bool empty = !fin && sl[k].key == kEncEmpty;
      r = hit ? sl[k].row : r;
      fin = fin || hit || empty;
    }
    if (fin) return r;
    h = (h + kProbeBatch) & t.cap_mask;
  }
  return -1;
}

__device__ inline int64_t idmap_lookup(const TableDev& t, unsigned long long e) {
  return idmap_lookup_at(t, e, idmap_hash(e) & t.cap_mask, 0);
}

// Claim the slot of an encoded key (its own if present, else the first empty
// one on its probe sequence); returns the slot index or -1 if the table is
// full.  Reads kProbeBatch slot keys per round trip; a stale read of an
// empty slot only costs a failed compare-and-swap (slots are never emptied
// during a call, so a slot read as occupied stays occupied).
__device__ inline int64_t idmap_claim(const TableDev& t, unsigned long long e) {
  uint64_t h = idmap_hash(e) & t.cap_mask;
  for (uint64_t probed = 0; probed <= t.cap_mask; probed += kProbeBatch) {
    unsigned long long k[kProbeBatch];
#pragma unroll
    for (int q = 0; q < kProbeBatch; ++q) k[q] = t.slots[(h + q) & t.cap_mask].key;
    for (int q = 0; q < kProbeBatch; ++q) {
      const uint64_t hq = (h + q) & t.cap_mask;
      if (k[q] == e) return static_cast<int64_t>(hq);
      if (k[q] == kEncEmpty) {
        const unsigned long long old = atomicCAS(&t.slots[hq].key, kEncEmpty, e);
        if (old == kEncEmpty || old == e) return static_cast<int64_t>(hq);
      }
    }
    h = (h + kProbeBatch) & t.cap_mask;
  }
  return -1;
}

// Slot of an encoded key in the scratch set: read first, compare-and-swap only
// an empty slot (a hot key, already present, costs no atomic here).
__device__ inline int64_t scratch_claim(const Scratch& sc, unsigned long long e) {
  uint64_t h = scratch_hash(e) & sc.mask;
  for (uint64_t probed = 0; probed <= sc.mask; ++probed) {
    unsigned long long cur = sc.slot[h].key;
    if (cur == kEncEmpty) cur = atomicCAS(&sc.slot[h].key, kEncEmpty, e);
    if (cur == kEncEmpty || cur == e) return static_cast<int64_t>(h);
    h = (h + 1) & sc.mask;
  }
  return -1;
}

// Exclusive block scan of five values per thread at once (two barriers).
template <int NT>
__device__ inline void block_excl_scan5(const int (&v)[5], int (&ex)[5], int (&tot)[5], int (*sh)[5]) {
  const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
  int inc[5];
#pragma unroll
  for (int a = 0; a < 5; ++a) inc[a] = wave_incl_scan(v[a]);
  if (lane == kWave - 1) {
#pragma unroll
    for (int a = 0; a < 5; ++a) sh[wid][a] = inc[a];
  }
  __syncthreads();
  if (threadIdx.x < 5) {
    const int a = threadIdx.x;
    int run = 0;
    for (int w = 0; w < NT / kWave; ++w) {
      const int t = sh[w][a];
      sh[w][a] = run;
      run += t;
    }
    sh[NT / kWave][a] = run;
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    ex[a] = sh[wid][a] + inc[a] - v[a];
    tot[a] = sh[NT / kWave][a];
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// pass 1: tile-local dedup in LDS, then the global scratch set
// ---------------------------------------------------------------------------

template <int NT>
__global__ __launch_bounds__(NT) void k_dedup_local(const int64_t* __restrict__ values, int64_t n, Scratch sc,
                                                        int32_t* __restrict__ slot_of, int32_t* __restrict__ occ_rank,
                                                        int* err) {
  constexpr int TILE = NT * kDedupItems;  // occurrences per block
  constexpr int SLOTS = 2 * TILE;         // LDS hash slots (load <= 0.5)
  // lkey: the key, then (read only by the slot's owner in between) its
  // scratch slot; lcnt: the count, then the global rank base of the tile's
  // occurrences of the key
  __shared__ unsigned long long lkey[SLOTS];
  __shared__ unsigned int lmin[SLOTS];
  __shared__ unsigned int lcnt[SLOTS];
  __shared__ short ldense[TILE];  // the tile's distinct keys: dense index -> LDS slot
  __shared__ int sh[NT / kWave + 1];
  const int tid = threadIdx.x;
  for (int s = tid; s < SLOTS; s += NT) {
    lkey[s] = kEncEmpty;
    lmin[s] = 0xFFFFFFFFu;
    lcnt[s] = 0u;
  }
  // every load is issued before the first wait (n > 0: indices are clamped)
  const int64_t base = static_cast<int64_t>(blockIdx.x) * TILE;
  int64_t raw[kDedupItems];
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) raw[k] = values[min(base + k * NT + tid, n - 1)];
  __syncthreads();
  int ls[kDedupItems];
  unsigned int lr[kDedupItems];
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) {
    const int64_t i = base + k * NT + tid;
    const unsigned long long e = static_cast<unsigned long long>(raw[k]) ^ kSign;
    ls[k] = -1;
    lr[k] = 0;
    if (i >= n) continue;
    if (e <= kEncTomb) {
      atomicOr(err, kErrKey);
      continue;
    }
    unsigned int h = static_cast<unsigned int>(mix64(e) >> 40) & (SLOTS - 1);
    while (true) {  // at most TILE keys in twice as many slots: terminates
      const unsigned long long old = atomicCAS(&lkey[h], kEncEmpty, e);
      if (old == kEncEmpty || old == e) break;
      h = (h + 1) & (SLOTS - 1);
    }
    atomicMin(&lmin[h], static_cast<unsigned int>(i));
    lr[k] = atomicAdd(&lcnt[h], 1u);
    ls[k] = static_cast<int>(h);
  }
  __syncthreads();
  // Dense list of the occupied slots, so a wavefront's global phase runs as
  // few rounds as the tile has distinct keys per thread (not one per slot).
  constexpr int kOwn = SLOTS / NT;
  int occ = 0;
#pragma unroll
  for (int j = 0; j < kOwn; ++j) occ += lkey[tid * kOwn + j] != kEncEmpty;
  int d;
  int at = block_excl_scan<NT>(occ, sh, d);
#pragma unroll
  for (int j = 0; j < kOwn; ++j)
    if (lkey[tid * kOwn + j] != kEncEmpty) ldense[at++] = static_cast<short>(tid * kOwn + j);
  __syncthreads();
  // Global phase, each step issued for all of a thread's keys before its
  // results are waited for: read the key's scratch slot; claim it with a
  // compare-and-swap if empty (a hot key, already present, costs no atomic);
  // lower the stored first position if this tile's is smaller (it only ever
  // decreases, so a stale read errs on the side of the atomic); add the
  // tile's count, whose old value is the rank base of the tile's occurrences.
  constexpr int kPer = TILE / NT;
  int sl[kPer];
  unsigned long long ke[kPer];
  ScratchSlot cur[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int q = tid + r * NT;
    sl[r] = q < d ? ldense[q] : -1;
    ke[r] = sl[r] >= 0 ? lkey[sl[r]] : kEncEmpty;
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r) cur[r] = sc.slot[scratch_hash(ke[r]) & sc.mask];  // idle lanes: one shared line
  int64_t gs[kPer];
  unsigned long long old[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    old[r] = cur[r].key;
    if (sl[r] >= 0 && cur[r].key == kEncEmpty)
      old[r] = atomicCAS(&sc.slot[scratch_hash(ke[r]) & sc.mask].key, kEncEmpty, ke[r]);
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    gs[r] = -1;
    if (sl[r] < 0) continue;
    if (old[r] == ke[r] || old[r] == kEncEmpty) {
      gs[r] = static_cast<int64_t>(scratch_hash(ke[r]) & sc.mask);
      if (old[r] == kEncEmpty) cur[r].first = 0xFFFFFFFFu;  // claimed here: always take the atomicMin
    }
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    if (sl[r] < 0 || gs[r] >= 0) continue;
    gs[r] = scratch_claim(sc, ke[r]);  // collision: probe on (rare)
    cur[r].first = 0xFFFFFFFFu;
    if (gs[r] < 0) atomicOr(err, kErrScratch);
  }
  unsigned int mn[kPer], cn[kPer], gb[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    mn[r] = sl[r] >= 0 ? lmin[sl[r]] : 0u;
    cn[r] = sl[r] >= 0 ? lcnt[sl[r]] : 0u;
  }
#pragma unroll
  for (int r = 0; r < kPer; ++r)
    if (gs[r] >= 0 && cur[r].first > mn[r]) atomicMin(&sc.slot[gs[r]].first, mn[r]);
#pragma unroll
  for (int r = 0; r < kPer; ++r) gb[r] = gs[r] >= 0 ? atomicAdd(&sc.slot[gs[r]].cnt, cn[r]) : 0u;
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    if (sl[r] < 0) continue;
    lkey[sl[r]] = static_cast<unsigned long long>(gs[r]);
    lcnt[sl[r]] = gb[r];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) {
    const int64_t i = base + k * NT + tid;
    if (i >= n) continue;
    const int g = ls[k] >= 0 ? static_cast<int>(static_cast<long long>(lkey[ls[k]])) : -1;
    const bool cand = g >= 0 && lmin[ls[k]] == static_cast<unsigned int>(i);
    slot_of[i] = g < 0 ? -1 : (g | (cand ? kCandBit : 0));
    occ_rank[i] = g >= 0 ? static_cast<int>(lcnt[ls[k]] + lr[k]) : 0;
  }
}

// ---------------------------------------------------------------------------
// pass 2: first occurrences probe the IDMap; tile sums
// ---------------------------------------------------------------------------

__device__ inline void load4(const int32_t* __restrict__ p, int64_t i0, int64_t n, int (&v)[4]) {
  if (i0 + 4 <= n) {
    const int4 a = *reinterpret_cast<const int4*>(p + i0);
    v[0] = a.x;
    v[1] = a.y;
    v[2] = a.z;
    v[3] = a.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = (i0 + k < n) ? p[i0 + k] : -1;
  }
}

template <int NT>
__global__ __launch_bounds__(NT) void k_rank_probe(TableDev t, Scratch sc, int32_t* __restrict__ slot_of,
                                                   int64_t n, int32_t* __restrict__ bsum, int64_t ntiles,
                                                   int64_t* cscal) {
  __shared__ int sh[NT / kWave + 1][5];
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * NT * kRankItems + threadIdx.x * kRankItems;
  int s[4];
  load4(slot_of, i0, n, s);
  // every load of a step is issued before its results are waited for: the
  // scratch slots of the tile-local firsts (other lanes read one shared
  // slot), then the first IDMap probe batch of every first occurrence
  bool f[4];
  ScratchSlot ss[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const bool cand = s[k] >= 0 && (s[k] & kCandBit);
    ss[k] = sc.slot[cand ? (s[k] & kSlotMask) : 0];
    f[k] = cand;
  }
  int c = 0, cf = 0, nl = 0, nu = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    f[k] = f[k] && ss[k].first == static_cast<unsigned int>(i0 + k);
    if (f[k]) {
      const int ck = static_cast<int>(ss[k].cnt);
      cf += 1;
      c += ck;
      if (ck > kLong) {
        nl += 1;
        nu += unit_count(ck);
      }
    }
  }
  uint64_t h[4];
  Slot pb[4][kProbeBatch];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[k] = f[k] ? idmap_hash(ss[k].key) & t.cap_mask : 0;
#pragma unroll
    for (int q = 0; q < kProbeBatch; ++q) pb[k][q] = t.slots[(h[k] + q) & t.cap_mask];
  }
  int nw = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (!f[k]) continue;
    int64_t r = -1;
    bool done = false;
#pragma unroll
    for (int q = 0; q < kProbeBatch; ++q) {  // selects only: the batch stays in registers
      const bool hit = !done && pb[k][q].key == ss[k].key;
      const bool empty = !done && pb[k][q].key == kEncEmpty;
      r = hit ? pb[k][q].row : r;
      done = done || hit || empty;
    }
    if (!done) r = idmap_lookup_at(t, ss[k].key, (h[k] + kProbeBatch) & t.cap_mask, kProbeBatch);
    ScratchAux* ax = &sc.aux[s[k] & kSlotMask];
    ax->row = r;
    ax->count = static_cast<int>(ss[k].cnt);
    nw += r < 0;
  }
  // the first occurrences are marked so the next pass reads only their keys
  if (cf) {
    if (i0 + 4 <= n) {
      *reinterpret_cast<int4*>(slot_of + i0) = make_int4(f[0] ? s[0] | kFirstBit : s[0], f[1] ? s[1] | kFirstBit : s[1],
                                                          f[2] ? s[2] | kFirstBit : s[2], f[3] ? s[3] | kFirstBit : s[3]);
    } else {
      for (int k = 0; k < 4 && i0 + k < n; ++k)
        if (f[k]) slot_of[i0 + k] = s[k] | kFirstBit;
    }
  }
  const int v[5] = {cf, c, nw, nl, nu};
  int ex[5], tot[5];
  block_excl_scan5<NT>(v, ex, tot, sh);
  if (threadIdx.x == 0) {
#pragma unroll
    for (int a = 0; a < 5; ++a) bsum[a * ntiles + blockIdx.x] = tot[a];
    if (blockIdx.x == 0) cscal[kCScanDone] = 0;  // the scan's completion counter
  }
}

// ---------------------------------------------------------------------------
// one-block scan of the five tile-sum arrays; row reservation
// ---------------------------------------------------------------------------

__device__ inline void publish_live(int64_t* h_live, int64_t tag, int64_t live) {
  // one 8-byte store to pinned host memory: (call tag << 48) | live rows
  if (h_live) {
    *reinterpret_cast<volatile int64_t*>(h_live) = (tag << 48) | live;
    __threadfence_system();
  }
}

// Scan of the five tile-sum arrays: block c scans chunk c (kScanChunk tiles,
// R per thread) in place and stores the chunk's totals; the last block to
// finish (a counter, no waiting) scans the chunk totals in place, reserves
// the rows of the new keys and publishes the live count.  A tile's prefix is
// then bsum[a][tile] + csum[a][tile / kScanChunk].
template <int R>
__global__ __launch_bounds__(1024) void k_scan5(int32_t* __restrict__ bsum, int64_t nb, int64_t ntiles,
                                                int32_t* __restrict__ csum, int64_t nch, int64_t* cscal,
                                                int64_t* tscal, int64_t* h_live, int64_t tag) {
  static_assert(1024 * R == kScanChunk, "one chunk per block");
  __shared__ int sh[1024 / kWave + 1][5];
  __shared__ bool last;
  const int64_t c = blockIdx.x;
  const int64_t lo = c * kScanChunk + static_cast<int64_t>(threadIdx.x) * R;
  int v[5][R];
#pragma unroll
  for (int a = 0; a < 5; ++a)
#pragma unroll
    for (int j = 0; j < R; ++j) v[a][j] = lo + j < nb ? bsum[a * ntiles + lo + j] : 0;
  int local[5], ex[5], tot[5];
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    local[a] = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) local[a] += v[a][j];
  }
  block_excl_scan5<1024>(local, ex, tot, sh);
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    int run = ex[a];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      if (lo + j < nb) bsum[a * ntiles + lo + j] = run;
      run += v[a][j];
    }
  }
  if (threadIdx.x == 0) {
#pragma unroll
    for (int a = 0; a < 5; ++a) csum[a * nch + c] = tot[a];
    __threadfence();
    const unsigned long long done =
        atomicAdd(reinterpret_cast<unsigned long long*>(&cscal[kCScanDone]), 1ull);
    last = done == static_cast<unsigned long long>(nch - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  // the last block: exclusive scan of the chunk totals (nch <= 1024 R)
  int cv[5][R];
  const int64_t clo = static_cast<int64_t>(threadIdx.x) * R;
#pragma unroll
  for (int a = 0; a < 5; ++a)
#pragma unroll
    for (int j = 0; j < R; ++j)
      cv[a][j] = clo + j < nch ? __hip_atomic_load(&csum[a * nch + clo + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    local[a] = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) local[a] += cv[a][j];
  }
  block_excl_scan5<1024>(local, ex, tot, sh);
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    int run = ex[a];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      if (clo + j < nch) csum[a * nch + clo + j] = run;
      run += cv[a][j];
    }
  }
  if (threadIdx.x != 0) return;
  cscal[kCScanDone] = 0;  // ready for the next call on this workspace
  cscal[kCU] = tot[0];
  cscal[kCValid] = tot[1];
  cscal[kCNewReq] = tot[2];
  cscal[kCNLong] = tot[3];
  cscal[kCNUnits] = tot[4];
  const int64_t live = tscal[kTLive];
  const int64_t lim = min(tscal[kTLimit], tscal[kTRowCap]);
  const int64_t room = lim > live ? lim - live : 0;
  const int64_t ins = tot[2] < room ? tot[2] : room;
  cscal[kCNew] = ins;
  cscal[kCBaseLive] = live;
  cscal[kCTrunc] = tot[2] > room ? 1 : 0;
  tscal[kTLive] = live + ins;
  publish_live(h_live, tag, live + ins);
}

// After the host grew the table: reserve again from the same live count.
__global__ void k_rereserve(int64_t* cscal, int64_t* tscal, int64_t* h_live, int64_t tag) {
  const int64_t live = cscal[kCBaseLive], req = cscal[kCNewReq];
  const int64_t lim = min(tscal[kTLimit], tscal[kTRowCap]);
  const int64_t room = lim > live ? lim - live : 0;
  const int64_t ins = req < room ? req : room;
  cscal[kCNew] = ins;
  cscal[kCTrunc] = req > room ? 1 : 0;
  tscal[kTLive] = live + ins;
  publish_live(h_live, tag, live + ins);
}

__global__ void k_zero_scalars(int64_t* cscal) { cscal[threadIdx.x] = 0; }

__global__ void k_scratch_clear(ScratchSlot* slots, int64_t n) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock)
    slots[i] = ScratchSlot{kEncEmpty, 0xFFFFFFFFu, 0u};
}

hipError_t launch_scratch_clear(ScratchSlot* slots, int64_t n, hipStream_t s) {
  k_scratch_clear<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(slots, n);
  return hipGetLastError();
}

hipError_t launch_rereserve(const Work& w, const TableDev& t, int64_t* h_live, int64_t tag, hipStream_t s) {
  k_rereserve<<<1, 1, 0, s>>>(w.scal, t.scal, h_live, tag);
  return hipGetLastError();
}

hipError_t launch_dedup_probe(const int64_t* values, int64_t n, const Scratch& sc, const TableDev& t, const Work& w,
                              int64_t* h_live, int64_t tag, hipEvent_t* ev_local, hipEvent_t* ev_probe,
                              hipStream_t s) {
  if (n <= 0) {
    k_zero_scalars<<<1, kCScalars, 0, s>>>(w.scal);
    return hipGetLastError();
  }
  const int64_t nb = (n + kRankTile - 1) / kRankTile;
  if (ev_local && ev_local[0]) (void)hipEventRecord(ev_local[0], s);
  k_dedup_local<kDedupThreads><<<grid_for(n, kDedupThreads * kDedupItems, 1ll << 31), kDedupThreads, 0, s>>>(
      values, n, sc, w.slot_of, w.occ_rank,
                                                                     reinterpret_cast<int*>(t.scal + kTErr));
  if (ev_local && ev_local[1]) (void)hipEventRecord(ev_local[1], s);
  if (ev_probe && ev_probe[0]) (void)hipEventRecord(ev_probe[0], s);
  k_rank_probe<kBlock><<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, sc, w.slot_of, n, w.bsum, w.ntiles,
                                                                   w.scal);
  if (ev_probe && ev_probe[1]) (void)hipEventRecord(ev_probe[1], s);
  const int64_t nch = (nb + kScanChunk - 1) / kScanChunk;
  k_scan5<kScanChunk / 1024><<<static_cast<unsigned>(nch), 1024, 0, s>>>(w.bsum, nb, w.ntiles, w.csum, nch, w.scal,
                                                                          t.scal, h_live, tag);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pass 3: unique ids, segments, rows, IDMap inserts
// ---------------------------------------------------------------------------

template <int NT>
__global__ __launch_bounds__(NT) void k_compact_insert(TableDev t, Scratch sc, Work w,
                                                       const int64_t* __restrict__ values, int64_t n) {
  __shared__ int sh[NT / kWave + 1][5];
  const int64_t i0 = static_cast<int64_t>(blockIdx.x) * NT * kRankItems + threadIdx.x * kRankItems;
  const int b = blockIdx.x;
  int pre[5];  // the tile's exclusive prefixes (first, count, new, hot, units)
  const int64_t nch = (static_cast<int64_t>(gridDim.x) + kScanChunk - 1) / kScanChunk;
#pragma unroll
  for (int a = 0; a < 5; ++a) pre[a] = w.bsum[a * w.ntiles + b] + w.csum[a * nch + b / kScanChunk];
  int s[4];
  load4(w.slot_of, i0, n, s);
  bool f[4];
  ScratchAux ax0[4];
  int cf = 0, cc = 0, cn = 0, cl = 0, cu = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    f[k] = s[k] >= 0 && (s[k] & kFirstBit);
    s[k] &= kSlotMask;
    ax0[k] = sc.aux[f[k] ? s[k] : 0];  // all four reads in flight together
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    cf += f[k];
    cc += f[k] ? ax0[k].count : 0;
    cn += (f[k] && ax0[k].row < 0);
    if (f[k] && ax0[k].count > kLong) {
      cl += 1;
      cu += unit_count(ax0[k].count);
    }
  }
  // the tile's first occurrences get consecutive unique ids, segments, rows
  // of new keys, hot-key indices and backward units
  const int v[5] = {cf, cc, cn, cl, cu};
  int ex[5], tot[5];
  block_excl_scan5<NT>(v, ex, tot, sh);
  int uid = pre[0] + ex[0];
  int start = pre[1] + ex[1];
  int64_t nr = pre[2] + ex[2];
  int lnext = pre[3] + ex[3];
  int unext = pre[4] + ex[4];
  const int64_t inserted = w.scal[kCNew];
  const int64_t live0 = w.scal[kCBaseLive];
  if (blockIdx.x == 0 && threadIdx.x == 0 && w.scal[kCTrunc]) atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrFull);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (!f[k]) continue;
    const int c = ax0[k].count;
    const unsigned long long ekey = static_cast<unsigned long long>(values[i0 + k]) ^ kSign;
    w.unique[uid] = values[i0 + k];
    int li = -1, ush = 0;
    if (c > kLong) {
      li = lnext++;
      ush = unit_shift(c);
      w.long_u[li] = uid;
      w.long_start[li] = unext;
      unext += unit_count(c);
    }
    int64_t row = ax0[k].row;
    if (row < 0) {
      if (nr < inserted) {
        const int64_t slot = idmap_claim(t, ekey);
        if (slot >= 0) {
          row = live0 + nr;
          t.slots[slot].row = row;
          w.new_list[nr] = uid;
        } else {
          atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
        }
      }
      ++nr;
    }
    w.rows[uid] = row;
    w.useg[uid] = Seg{row, start, c};
    ScratchAux ax;
    ax.row = row;
    ax.start = start;
    ax.uid = uid;
    ax.count = c;
    ax.long_idx = li;
    ax.unit_shift = ush;
    ax.pad = 0;
    sc.aux[s[k]] = ax;
    ++uid;
    start += c;
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

// Lane groups of 16 write the rows of the inserted keys: w from the init
// formula, optimizer state zero, 16 bytes per lane per store.  Block `blk`
// of `nblk` takes every nblk-th group of keys.
__device__ inline void init_rows(const TableDev& t, const Work& w, int64_t blk, int64_t nblk) {
  constexpr int G = 16;
  const int lane = threadIdx.x % G, grp = threadIdx.x / G;
  const int64_t inserted = w.scal[kCNew];
  const int chunks = static_cast<int>(t.store.stride / 16);
  const int wbytes = t.dim * (t.row_dtype ? 2 : 4);
  for (int64_t q = blk * (kBlock / G) + grp; q < inserted; q += nblk * (kBlock / G)) {
    const int u = w.new_list[q];
    const int64_t row = w.useg[u].row;
    const uint64_t z = mix64(static_cast<uint64_t>(w.unique[u]) ^ mix64(t.seed));
    uint8_t* rp = t.store.row(row);
    for (int ch = lane; ch < chunks; ch += G) {
      const int off = ch * 16;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (off < wbytes) {
        if (t.row_dtype == 0) {
          const int j0 = off / 4;
          val = make_uint4(__float_as_uint(init_value(z, j0, t.lo, t.span)),
                           __float_as_uint(init_value(z, j0 + 1, t.lo, t.span)),
                           __float_as_uint(init_value(z, j0 + 2, t.lo, t.span)),
                           __float_as_uint(init_value(z, j0 + 3, t.lo, t.span)));
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

// The per-occurrence pass: inverse[i] = unique id of occurrence i (-1 for a
// rejected key), and the occurrence of rank 0 of each key returns its scratch
// slot to empty, so the scratch never needs a full clear.  For a forward
// (OCC) it also writes each occurrence's row and its position in the
// occurrence list, and the descriptor of every backward unit of a hot key.
template <bool OCC>
__device__ inline void occ_pass(const Scratch& sc, const Work& w, int64_t n, int64_t blk) {
  const int64_t i0 = (blk * kBlock + threadIdx.x) * 4;
  if (i0 >= n) return;
  int s[4], rk[4];
  load4(w.slot_of, i0, n, s);
  load4(w.occ_rank, i0, n, rk);
  ScratchAux a[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) a[k] = sc.aux[s[k] >= 0 ? (s[k] & kSlotMask) : 0];  // all in flight together
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (s[k] < 0) {
      a[k].row = -1;
      a[k].uid = -1;
      a[k].start = 0;
      a[k].long_idx = -1;
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (s[k] < 0 || i0 + k >= n) continue;
    if (rk[k] == 0) sc.slot[s[k] & kSlotMask] = ScratchSlot{kEncEmpty, 0xFFFFFFFFu, 0u};
    if (OCC && a[k].long_idx >= 0) {
      const int sh = a[k].unit_shift;
      const int usz = kUnit << sh;
      if ((rk[k] & (usz - 1)) == 0) {
        const int p = a[k].start + rk[k];
        w.units[w.long_start[a[k].long_idx] + (rk[k] >> (kUnitLog2 + sh))] =
            Unit{a[k].long_idx, p, min(p + usz, a[k].start + a[k].count), 0};
      }
    }
  }
  if (i0 + 4 <= n) {
    *reinterpret_cast<int4*>(w.inverse + i0) = make_int4(a[0].uid, a[1].uid, a[2].uid, a[3].uid);
    if (OCC) {
      *reinterpret_cast<longlong2*>(w.occ_row + i0) = make_longlong2(a[0].row, a[1].row);
      *reinterpret_cast<longlong2*>(w.occ_row + i0 + 2) = make_longlong2(a[2].row, a[3].row);
      *reinterpret_cast<int4*>(w.occ_pos + i0) =
          make_int4(s[0] >= 0 ? a[0].start + rk[0] : -1, s[1] >= 0 ? a[1].start + rk[1] : -1,
                    s[2] >= 0 ? a[2].start + rk[2] : -1, s[3] >= 0 ? a[3].start + rk[3] : -1);
    }
  } else {
    for (int k = 0; k < 4 && i0 + k < n; ++k) {
      w.inverse[i0 + k] = a[k].uid;
      if (OCC) {
        w.occ_row[i0 + k] = a[k].row;
        w.occ_pos[i0 + k] = s[k] >= 0 ? a[k].start + rk[k] : -1;
      }
    }
  }
}

// The last pass of a lookup: blocks [0, occ_blocks) run the per-occurrence
// pass, the others write the rows of the inserted keys (both only need the
// compaction, so they share one launch).
template <bool OCC>
__global__ __launch_bounds__(kBlock) void k_occ_init(Scratch sc, TableDev t, Work w, int64_t n, int64_t occ_blocks) {
  const int64_t b = blockIdx.x;
  if (b < occ_blocks) occ_pass<OCC>(sc, w, n, b);
  else init_rows(t, w, b - occ_blocks, static_cast<int64_t>(gridDim.x) - occ_blocks);
}

hipError_t launch_compact_insert(const int64_t* values, int64_t n, const Scratch& sc, const TableDev& t, const Work& w,
                                 bool occ_lists, hipEvent_t* ev_compact, hipEvent_t* ev_init, hipEvent_t* ev_occ,
                                 hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + kRankTile - 1) / kRankTile;
  if (ev_compact && ev_compact[0]) (void)hipEventRecord(ev_compact[0], s);
  k_compact_insert<kBlock><<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, sc, w, values, n);
  if (ev_compact && ev_compact[1]) (void)hipEventRecord(ev_compact[1], s);
  // one launch: the per-occurrence pass and the new rows (the init-rows and
  // occurrence events both bracket it)
  if (ev_init && ev_init[0]) (void)hipEventRecord(ev_init[0], s);
  if (ev_occ && ev_occ[0]) (void)hipEventRecord(ev_occ[0], s);
  const int64_t ob = grid_for(n, kBlock * 4, 1ll << 31);
  const int64_t ib = grid_for(n, kBlock / 16, 8192);
  if (occ_lists) k_occ_init<true><<<static_cast<unsigned>(ob + ib), kBlock, 0, s>>>(sc, t, w, n, ob);
  else k_occ_init<false><<<static_cast<unsigned>(ob + ib), kBlock, 0, s>>>(sc, t, w, n, ob);
  if (ev_occ && ev_occ[1]) (void)hipEventRecord(ev_occ[1], s);
  if (ev_init && ev_init[1]) (void)hipEventRecord(ev_init[1], s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// find-or-insert results, find-only lookups, rehash, export, read-back
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_map_rows(const int32_t* __restrict__ inverse, const int64_t* __restrict__ rows,
                                                     int64_t n, int64_t* __restrict__ out, const int64_t* cscal,
                                                     int64_t* n_inserted) {
  const int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x;
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
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const unsigned long long e = static_cast<unsigned long long>(keys[i]) ^ kSign;
    out[i] = e <= kEncTomb ? -1 : idmap_lookup(t, e);
  }
}

hipError_t launch_find(const TableDev& t, const int64_t* keys, int64_t n, int64_t* rows_out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_find<<<grid_for(n, kBlock, 16384), kBlock, 0, s>>>(t, keys, n, rows_out);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_rehash(const Slot* __restrict__ old, int64_t old_cap, TableDev t) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < old_cap;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
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
  for (int64_t i = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; i < cap_slots;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
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
  for (int64_t idx = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * kBlock) {
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
      for (int q = 0; q < t.nstate; ++q) state_out[(i * t.nstate + q) * t.dim + j] = ok ? sp[q * t.dim + j] : __builtin_nanf("");
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

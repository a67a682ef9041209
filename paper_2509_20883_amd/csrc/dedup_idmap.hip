// Dedup and IDMap kernels of the sparse embedding step (gfx950).
//
// RecIS keeps a two-tier store: an IDMap from feature id to an offset and
// Blocks holding the rows ("Optimization for Memory Bound"); ids are
// deduplicated before the lookup ("ids partition").  The dedup gives the
// unique keys in first-occurrence order.  It uses no global atomics (on this
// GPU they serialise at the memory side): keys are grouped by a hash
// partition instead, so every key is counted by exactly one block in LDS.
//   k_tile_dedup     per block, consecutive tiles of 4096 occurrences: LDS
//                    dedup; one record per distinct key of a tile (key, first
//                    position and count in the tile), the tile's records in
//                    the order of their first positions; at the end the block
//                    copies its records into partition order
//   k_part_dedup     one block per partition, reading its records from every
//                    dedup block: LDS dedup (first position = min, count =
//                    sum, rank base of each record), the key's IDMap probe;
//                    the key's first record is flagged
//   k_first_sums     per tile of records: sums over the first records (keys,
//                    counts, keys not found, hot keys, backward units); the
//                    records, tile after tile, list each key once in the
//                    order of its first position
//   k_scan5          scan of those tile sums; reserves the rows of new keys
//   k_compact        unique ids in first-occurrence order, occurrence-list
//                    segments, rows; new keys claim an IDMap slot
//   k_occ_init       per occurrence: unique id (inverse), row, position in the
//                    occurrence list, hot-key backward units.  Its other
//                    blocks write the initial rows of the new keys
#include "device_common.h"

#include <algorithm>

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
  if (wid == 0) {  // one wave scans the per-wave totals of each value
    static_assert(NT / kWave <= kWave, "one wave scans the per-wave totals");
#pragma unroll
    for (int a = 0; a < 5; ++a) {
      const int t = lane < NT / kWave ? sh[lane][a] : 0;
      const int i2 = wave_incl_scan(t);
      if (lane < NT / kWave) sh[lane][a] = i2 - t;
      if (lane == kWave - 1) sh[NT / kWave][a] = i2;
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < 5; ++a) {
    ex[a] = sh[wid][a] + inc[a] - v[a];
    tot[a] = sh[NT / kWave][a];
  }
  __syncthreads();
}

__device__ inline uint32_t part_of(unsigned long long e, int logP) {
  return logP == 0 ? 0u : static_cast<uint32_t>(part_hash(e) >> (64 - logP));
}

// ---------------------------------------------------------------------------
// pass 1: tile dedup in LDS; one record per distinct key of a tile
// ---------------------------------------------------------------------------

// A dedup block whose records fill at most this many LDS chunks (8192
// records each) writes their partition-order copy with coalesced stores.
constexpr int kStageChunks = 4;

template <int NT>
__global__ __launch_bounds__(NT) void k_tile_dedup(const int64_t* __restrict__ values, int64_t n, Work w, int* err) {
  constexpr int TILE = NT * kDedupItems;
  constexpr int SLOTS = 2 * TILE;  // LDS hash slots (load <= 0.5)
  static_assert(TILE == kDedupTile, "tile size");
  // One LDS buffer: the hash table while the tiles are deduplicated (slot
  // keys; lmin: the key's first position in the tile, then its record
  // index; lcnt: its count), then the staging buffer of the partition-order
  // copy (one 16-byte record per slot).
  __shared__ TileRec lbuf[SLOTS];
  unsigned long long* const lkey = reinterpret_cast<unsigned long long*>(lbuf);
  unsigned int* const lmin = reinterpret_cast<unsigned int*>(lkey + SLOTS);
  unsigned int* const lcnt = lmin + SLOTS;
  __shared__ short ldense[TILE];          // the tile's distinct keys: dense index -> LDS slot
  __shared__ unsigned int lpc[kMaxParts];  // the block's records per partition
  __shared__ int sh[NT / kWave + 1];
  __shared__ int lfirst[kDedupItems * (NT / kWave) + 1];  // first occurrences per (item, wave), then their prefix
  const FrontGeom g = w.g;
  const int tid = threadIdx.x;
  const int64_t blk = blockIdx.x;
  for (int q = tid; q < g.P; q += NT) lpc[q] = 0u;
  if (blk == 0 && tid == 0) w.scal[kCScanDone] = 0;  // completion counter of this call's scan
  const int64_t t0 = blk * g.R;
  const int64_t t1 = min(t0 + g.R, g.ntiles);
  TileRec* rec = w.trec + blk * g.rcap;
  // the next tile's ids are loaded while this one is processed (n > 0:
  // indices are clamped)
  int64_t nxt[kDedupItems];
#pragma unroll
  for (int k = 0; k < kDedupItems; ++k) nxt[k] = values[min(t0 * TILE + k * NT + tid, n - 1)];
  unsigned int nrec = 0;
  for (int64_t tile = t0; tile < t1; ++tile) {
    const int64_t base = tile * TILE;
    int64_t raw[kDedupItems];
#pragma unroll
    for (int k = 0; k < kDedupItems; ++k) raw[k] = nxt[k];
    if (tile + 1 < t1) {
#pragma unroll
      for (int k = 0; k < kDedupItems; ++k) nxt[k] = values[min(base + TILE + k * NT + tid, n - 1)];
    }
    if (tile == t0) {  // later tiles find the table cleared by their predecessor
      for (int q = tid; q < SLOTS; q += NT) {
        lkey[q] = kEncEmpty;
        lmin[q] = 0xFFFFFFFFu;
        lcnt[q] = 0u;
      }
    }
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
    // dense list of the tile's keys in the order of their first positions:
    // the first occurrences (lmin of the slot is the position itself), ranked
    // in position order (item k of thread tid is position base + k*NT + tid:
    // item-major, then wave, then lane)
    int d;
    {
      constexpr int NW = NT / kWave;
      const int lane = tid & (kWave - 1), wid = tid / kWave;
      const uint64_t below = (1ull << lane) - 1ull;
      bool fst[kDedupItems];
      uint64_t bal[kDedupItems];
#pragma unroll
      for (int k = 0; k < kDedupItems; ++k) {
        const int64_t i = base + k * NT + tid;
        fst[k] = ls[k] >= 0 && lmin[ls[k]] == static_cast<unsigned int>(i);
        bal[k] = __ballot(fst[k]);
        if (lane == 0) lfirst[k * NW + wid] = __popcll(bal[k]);
      }
      __syncthreads();
      if (tid < kWave) {  // exclusive prefix over (item, wave) in position order: one wave's scan
        static_assert(kDedupItems * NW <= kWave, "one wave scans the (item, wave) counts");
        const int c = tid < kDedupItems * NW ? lfirst[tid] : 0;
        const int inc = wave_incl_scan(c);
        if (tid < kDedupItems * NW) lfirst[tid] = inc - c;
        if (tid == kWave - 1) lfirst[kDedupItems * NW] = inc;
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < kDedupItems; ++k)
        if (fst[k]) ldense[lfirst[k * NW + wid] + __popcll(bal[k] & below)] = static_cast<short>(ls[k]);
      d = lfirst[kDedupItems * NW];
    }
    __syncthreads();
    // one record per distinct key (nrec + d <= the block's occurrences <= rcap)
    for (int q = tid; q < d; q += NT) {
      const int sl = ldense[q];
      const unsigned long long e = lkey[sl];
      const unsigned int pr = atomicAdd(&lpc[part_of(e, g.logP)], 1u);
      rec[nrec + q] = TileRec{e, lmin[sl], (pr << 12) | (lcnt[sl] - 1u)};
      lmin[sl] = nrec + static_cast<unsigned int>(q);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kDedupItems; ++k) {
      const int64_t i = base + k * NT + tid;
      if (i >= n) continue;
      // read again only by the passes after the compaction: non-temporal
      __builtin_nontemporal_store(ls[k] < 0 ? kOccRejected : ((lmin[ls[k]] << 12) | lr[k]), &w.occ_word[i]);
    }
    nrec += static_cast<unsigned int>(d);
    __syncthreads();
    // empty the occupied slots for the next tile
    for (int q = tid; q < d; q += NT) {
      const int sl = ldense[q];
      lkey[sl] = kEncEmpty;
      lmin[sl] = 0xFFFFFFFFu;
      lcnt[sl] = 0u;
    }
  }
  if (tid == 0) w.nrec[blk] = static_cast<int>(nrec);
  // the block's records per partition and their offsets in partition order
  // (in place in lpc), then the partition-ordered copy of the records
  constexpr int PPT = kMaxParts / NT;
  int c[PPT];
  int loc = 0;
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    const int q = tid * PPT + j;
    c[j] = q < g.P ? static_cast<int>(lpc[q]) : 0;
    loc += c[j];
  }
  int tot;
  int run = block_excl_scan<NT>(loc, sh, tot);
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    const int q = tid * PPT + j;
    if (q < g.P) {
      w.pcnt[blk * g.P + q] = c[j];
      w.poff[blk * g.P + q] = run;
      lpc[q] = static_cast<unsigned int>(run);
    }
    run += c[j];
  }
  __syncthreads();
  TileRec* srt = w.srec + blk * g.rcap;
  constexpr int U8 = 8;  // records in flight per thread
  // Record j goes to position lpc[partition] + its rank in the partition.
  // A block of at most kStageChunks chunks of SLOTS records assembles each
  // chunk in LDS (every pass reads all of the block's records again) and
  // writes it out with coalesced full-line stores; a larger block scatters
  // the records (runs of a few 16-byte records per partition: partial-line
  // writes, costly once the copies outgrow the memory-side cache).
  const unsigned int chunks = (nrec + SLOTS - 1) / SLOTS;
  const bool staged = chunks <= static_cast<unsigned int>(kStageChunks);
  for (unsigned int ch = 0; ch < (staged ? chunks : 1u); ++ch) {
    const unsigned int o0 = ch * SLOTS;
    const unsigned int o1 = min(o0 + static_cast<unsigned int>(SLOTS), nrec);
    for (unsigned int j0 = tid; j0 < nrec; j0 += U8 * NT) {
      TileRec r[U8];
#pragma unroll
      for (int u = 0; u < U8; ++u) {
        const unsigned int j = j0 + u * NT;
        if (j < nrec) r[u] = rec[j];
      }
#pragma unroll
      for (int u = 0; u < U8; ++u) {
        const unsigned int j = j0 + u * NT;
        if (j >= nrec) continue;
        const unsigned int o = lpc[part_of(r[u].key, g.logP)] + (r[u].meta >> 12);
        const TileRec x{r[u].key, r[u].tmin, (j << 12) | (r[u].meta & 0xFFFu)};
        if (!staged) srt[o] = x;
        else if (o >= o0 && o < o1) lbuf[o - o0] = x;
      }
    }
    if (staged) {
      __syncthreads();
      for (unsigned int o = o0 + tid; o < o1; o += NT) srt[o] = lbuf[o - o0];
      __syncthreads();  // the next chunk reuses the buffer
    }
  }
}

// ---------------------------------------------------------------------------
// pass 2: one block per partition: LDS dedup of its records, IDMap probe
// ---------------------------------------------------------------------------

// Resolve a probe batch read at the key's home slot; continue the probe if
// the batch neither holds the key nor an empty slot.
__device__ inline int64_t resolve_probe(const TableDev& t, unsigned long long e, uint64_t h,
                                        const Slot (&pb)[kProbeBatch]) {
  int64_t r = -1;
  bool done = false;
#pragma unroll
  for (int q = 0; q < kProbeBatch; ++q) {  // selects only: the batch stays in registers
    const bool hit = !done && pb[q].key == e;
    const bool empty = !done && pb[q].key == kEncEmpty;
    r = hit ? pb[q].row : r;
    done = done || hit || empty;
  }
  if (!done) r = idmap_lookup_at(t, e, (h + kProbeBatch) & t.cap_mask, kProbeBatch);
  return r;
}

// The partition's records are read from every dedup block's
// partition-ordered copy (segment b: cnt[b] records at off[b]).  A key's
// index is the position of its first record (the one holding its first
// position): for a lookup its tile-order position, so the key info of a
// tile's first records lies together, in the order in which the
// first-occurrence sums and the compaction read and write it, and the info
// of a key seen once lies beside its ids' records; for the ids partition
// (no key info) its position in the partition-ordered copy, whose entry
// there holds the key.
// A partition of at most kPartSlots records is done in one pass with each
// thread's records in registers (its distinct keys always fit the table);
// a larger one in sweeps of at most kPartSweep records by a hash of the key,
// and if a sweep's keys do not fit (a skewed hash) the partition starts
// again with twice as many sweeps.
__device__ inline void probe_store_keys(const TableDev& t, const Work& w, int64_t n, int d, const short* cdense,
                                        const unsigned long long* ckey, const unsigned long long* cfp,
                                        const unsigned int* ccnt) {
  constexpr int NT = kPartThreads;
  constexpr int KP = 4;  // keys per thread per round: their probe batches in flight together
  for (int q0 = 0; q0 < d; q0 += KP * NT) {
    int sl[KP];
    unsigned long long e[KP];
    uint64_t h[KP];
    Slot pb[KP][kProbeBatch];
#pragma unroll
    for (int u = 0; u < KP; ++u) {
      const int q = q0 + u * NT + static_cast<int>(threadIdx.x);
      sl[u] = q < d ? cdense[q] : -1;
      e[u] = sl[u] >= 0 ? ckey[sl[u]] : kEncEmpty;
      h[u] = sl[u] >= 0 ? (idmap_hash(e[u]) & t.cap_mask) : 0;  // idle lanes read one shared line
      if (t.slots) {
#pragma unroll
        for (int k = 0; k < kProbeBatch; ++k) pb[u][k] = t.slots[(h[u] + k) & t.cap_mask];
      }
    }
#pragma unroll
    for (int u = 0; u < KP; ++u) {
      if (sl[u] < 0) continue;
      const unsigned int kidx = static_cast<unsigned int>(cfp[sl[u]]);
      {
        KeyInfo ki;
        ki.row = t.slots ? resolve_probe(t, e[u], h[u], pb[u]) : 0;  // no table: nothing to probe
        ki.key = static_cast<long long>(e[u] ^ kSign);
        ki.count = static_cast<int>(ccnt[sl[u]]);
        ki.uid = -1;
        ki.start = 0;
        ki.long_idx = -1;
        w.kinfo[kidx] = ki;
      }
    }
  }
}

// Enter key e into the LDS table (linear probing from slot h).  Returns the
// slot, or -1 if every slot holds another key.
__device__ inline int lds_insert(unsigned long long* ckey, unsigned long long e, uint64_t hh) {
  constexpr int S = kPartSlots;
  unsigned int sl = static_cast<unsigned int>(hh >> 20) & (S - 1);
  for (int probes = 0; probes < S; ++probes) {
    const unsigned long long old = atomicCAS(&ckey[sl], kEncEmpty, e);
    if (old == kEncEmpty || old == e) return static_cast<int>(sl);
    sl = (sl + 1) & (S - 1);
  }
  return -1;
}

__global__ __launch_bounds__(kPartThreads) void k_part_dedup(TableDev t, Work w, int64_t n) {
  constexpr int NT = kPartThreads, S = kPartSlots, OWN = S / NT, K = kPartFast;
  constexpr int kMaxSweeps = 1 << 10;
  constexpr int BPT = (kMaxDedupBlocks + NT - 1) / NT;
  __shared__ unsigned long long ckey[S];
  // (first position << 32 | position of the record holding it): the minimum
  // over the key's records gives the key's first position and its key index
  __shared__ unsigned long long cfp[S];
  __shared__ unsigned int ccnt[S];
  __shared__ short cdense[S];  // dense index -> slot
  __shared__ int cpre[kMaxDedupBlocks];   // exclusive prefix of the segment sizes
  __shared__ int cbase[kMaxDedupBlocks];  // position of each segment
  __shared__ int sh[NT / kWave + 1];
  __shared__ int ovf;
  const FrontGeom g = w.g;
  const int tid = threadIdx.x;
  const int p = blockIdx.x;
  // the partition's segments (thread tid holds blocks tid*BPT ...)
  int cn[BPT];
  int loc = 0;
#pragma unroll
  for (int j = 0; j < BPT; ++j) {
    const int b = tid * BPT + j;
    cn[j] = b < g.nblk ? w.pcnt[static_cast<int64_t>(b) * g.P + p] : 0;
    if (b < g.nblk) cbase[b] = static_cast<int>(b * g.rcap) + w.poff[static_cast<int64_t>(b) * g.P + p];
    loc += cn[j];
  }
  int nr;
  int run = block_excl_scan<NT>(loc, sh, nr);
#pragma unroll
  for (int j = 0; j < BPT; ++j) {
    const int b = tid * BPT + j;
    if (b < g.nblk) cpre[b] = run;
    run += cn[j];
  }
  for (int q = tid; q < S; q += NT) {
    ckey[q] = kEncEmpty;
    cfp[q] = ~0ull;
    ccnt[q] = 0u;
  }
  if (tid == 0) ovf = 0;
  __syncthreads();
  if (nr == 0) return;  // the whole block
  const int nb = static_cast<int>(g.nblk);
  // position of the fr-th record of the partition: the last segment whose
  // prefix is <= fr (empty segments share their successor's prefix)
  auto rec_pos = [&](int fr) {
    int lo = 0, hi = nb;  // cpre[lo] <= fr; the answer is in [lo, hi)
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (cpre[mid] <= fr) lo = mid;
      else hi = mid;
    }
    return cbase[lo] + (fr - cpre[lo]);
  };
  // dense list of the occupied slots: thread tid owns slots tid + j * NT
  // (consecutive lanes, consecutive slots: no bank conflicts), read once
  static_assert(OWN <= 32, "occupancy mask");
  auto dense_list = [&]() {
    unsigned int om = 0u;
#pragma unroll
    for (int j = 0; j < OWN; ++j) om |= static_cast<unsigned int>(ckey[j * NT + tid] != kEncEmpty) << j;
    int d;
    int at = block_excl_scan<NT>(__popc(om), sh, d);
#pragma unroll
    for (int j = 0; j < OWN; ++j)
      if ((om >> j) & 1u) cdense[at++] = static_cast<short>(j * NT + tid);
    __syncthreads();
    return d;
  };

  // the key index a record would give its key (see above)
  auto rec_index = [&](int pos, const TileRec& x) {
    return w.kinfo ? static_cast<unsigned int>((pos / g.rcap) * g.rcap + (x.meta >> 12))
                   : static_cast<unsigned int>(pos);
  };
  bool fresh = true;  // the LDS table is clear
  if (nr <= NT * K) {
    // one pass: the thread's records tid, tid + NT, ... stay in registers
    // (up to kPartSlots records their keys always fit the table; beyond, a
    // full table sends the partition to the sweeps)
    int pos[K];
    TileRec x[K];
#pragma unroll
    for (int k = 0; k < K; ++k) pos[k] = tid + k * NT < nr ? rec_pos(tid + k * NT) : -1;
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (pos[k] >= 0) x[k] = w.srec[pos[k]];
    int sl[K];
    unsigned int rb[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      sl[k] = -1;
      rb[k] = 0;
      if (pos[k] < 0) continue;
      sl[k] = lds_insert(ckey, x[k].key, part_hash(x[k].key));
      if (sl[k] < 0) {
        ovf = 1;
        pos[k] = -1;
        continue;
      }
      atomicMin(&cfp[sl[k]], (static_cast<unsigned long long>(x[k].tmin) << 32) | rec_index(pos[k], x[k]));
      rb[k] = atomicAdd(&ccnt[sl[k]], (x[k].meta & 0xFFFu) + 1u);
    }
    __syncthreads();
    if (!ovf) {
      if (w.kinfo) {  // null (ids partition): no key info, no probe
        const int d = dense_list();
        probe_store_keys(t, w, n, d, cdense, ckey, cfp, ccnt);
      }
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (pos[k] < 0) continue;
        const int64_t src = (static_cast<int64_t>(pos[k]) / g.rcap) * g.rcap + (x[k].meta >> 12);
        const unsigned int kidx = static_cast<unsigned int>(cfp[sl[k]]);
        // the key's first record is the one whose index is its key index
        const unsigned int fl = kidx == rec_index(pos[k], x[k]) ? kRecFirst : 0u;
        w.recres[src] = make_int2(static_cast<int>(kidx), static_cast<int>(rb[k] | fl));
      }
      return;
    }
    fresh = false;
    __syncthreads();  // every thread has read ovf before the sweeps reset it
  }

  // sweeps (rare: a partition far above the average size)
  int nsw = min((nr + kPartSweep - 1) / kPartSweep, kMaxSweeps);
  int s = 0;
  while (s < nsw) {
    if (!fresh) {
      for (int q = tid; q < S; q += NT) {
        ckey[q] = kEncEmpty;
        cfp[q] = ~0ull;
        ccnt[q] = 0u;
      }
    }
    fresh = false;
    if (tid == 0) ovf = 0;
    __syncthreads();
    for (int fr = tid; fr < nr; fr += NT) {
      const int pos = rec_pos(fr);
      const TileRec x = w.srec[pos];
      const uint64_t h = part_hash(x.key);
      if (static_cast<int>((h & 0xFFFFFull) % static_cast<uint64_t>(nsw)) != s) continue;
      const int sl = lds_insert(ckey, x.key, h);
      if (sl < 0) {
        ovf = 1;
        continue;
      }
      atomicMin(&cfp[sl], (static_cast<unsigned long long>(x.tmin) << 32) | rec_index(pos, x));
      const unsigned int rb = atomicAdd(&ccnt[sl], (x.meta & 0xFFFu) + 1u);
      w.ptmp[pos] = make_int2(static_cast<int>(((x.meta >> 12) << 12) | static_cast<unsigned int>(sl)),
                              static_cast<int>(rb));
    }
    __syncthreads();
    if (ovf) {
      __syncthreads();  // every thread has read ovf
      if (nsw >= kMaxSweeps) {
        if (tid == 0) atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
        return;
      }
      nsw *= 2;
      s = 0;
      continue;
    }
    if (w.kinfo) {
      const int d = dense_list();
      probe_store_keys(t, w, n, d, cdense, ckey, cfp, ccnt);
    }
    for (int fr = tid; fr < nr; fr += NT) {
      const int pos = rec_pos(fr);
      const uint64_t h = part_hash(w.srec[pos].key);
      if (static_cast<int>((h & 0xFFFFFull) % static_cast<uint64_t>(nsw)) != s) continue;
      const int2 tp = w.ptmp[pos];
      const int64_t src = (static_cast<int64_t>(pos) / g.rcap) * g.rcap + (static_cast<uint32_t>(tp.x) >> 12);
      const unsigned int kidx = static_cast<unsigned int>(cfp[tp.x & 0xFFF]);
      const unsigned int ix = w.kinfo ? static_cast<unsigned int>(src) : static_cast<unsigned int>(pos);
      const unsigned int fl = kidx == ix ? kRecFirst : 0u;
      w.recres[src] = make_int2(static_cast<int>(kidx), static_cast<int>(static_cast<unsigned int>(tp.y) | fl));
    }
    ++s;
    __syncthreads();  // the next sweep clears the LDS
  }
}

// ---------------------------------------------------------------------------
// pass 5: tile sums over the first occurrences
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

// Key info of key index k (k >= 0), or of index 0 for an idle lane (read,
// never used: every load of a step is issued before its results are waited for).
__device__ inline KeyInfo key_info(const Work& w, int k) {
  return w.kinfo[min(max(k, 0), static_cast<int>(w.nkeyidx - 1))];
}

// The first records of record tile rt (4 record slots per thread): the key
// index of each first record (a key's first record is its only one that is
// counted), or -1.  Records past the dedup block's count are not read.
__device__ inline void first_records(const Work& w, int64_t rt, int (&f)[4]) {
  const int64_t per = w.g.rcap / kRankTile;  // record tiles per dedup block
  const int64_t blk = rt / per;
  const int64_t r0 = (rt % per) * kRankTile + static_cast<int64_t>(threadIdx.x) * 4;
  const int64_t nr = w.nrec[blk];
  const int4 a = *reinterpret_cast<const int4*>(w.recres + blk * w.g.rcap + r0);  // 2 records
  const int4 b = *reinterpret_cast<const int4*>(w.recres + blk * w.g.rcap + r0 + 2);
  const int x[4] = {a.x, a.z, b.x, b.z}, y[4] = {a.y, a.w, b.y, b.w};
#pragma unroll
  for (int k = 0; k < 4; ++k)
    f[k] = r0 + k < nr && (static_cast<uint32_t>(y[k]) & kRecFirst) ? x[k] : -1;
}

// Record tile rt lies wholly past its dedup block's records (a block's record
// slots are sized for its ids, and distinct keys are fewer).
__device__ inline bool empty_record_tile(const Work& w, int64_t rt) {
  const int64_t per = w.g.rcap / kRankTile;
  return (rt % per) * kRankTile >= w.nrec[rt / per];
}

// Per record tile: sums over its first records (keys, their counts, keys not
// found, hot keys, hot-key units).  Record tiles in block-major order list
// the keys in the order of their first positions.
template <int NT>
__global__ __launch_bounds__(NT) void k_first_sums(Work w) {
  __shared__ int sh[NT / kWave + 1][5];
  if (empty_record_tile(w, blockIdx.x)) {  // block-uniform
    if (threadIdx.x < 5) w.bsum[threadIdx.x * w.ntiles + blockIdx.x] = 0;
    return;
  }
  int f[4];
  first_records(w, blockIdx.x, f);
  KeyInfo ki[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) ki[k] = key_info(w, f[k]);
  int cf = 0, c = 0, nw = 0, nl = 0, nu = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (f[k] < 0) continue;
    cf += 1;
    c += ki[k].count;
    nw += ki[k].row < 0;
    if (ki[k].count > kLong) {
      nl += 1;
      nu += unit_count(ki[k].count);
    }
  }
  const int v[5] = {cf, c, nw, nl, nu};
  int ex[5], tot[5];
  block_excl_scan5<NT>(v, ex, tot, sh);
  if (threadIdx.x == 0) {
#pragma unroll
    for (int a = 0; a < 5; ++a) w.bsum[a * w.ntiles + blockIdx.x] = tot[a];
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

// Rows for `req` keys not found, from `hw` rows allocated, `keys` live keys
// and `F` free rows: as many as both the IDMap (its key limit counts the
// tombstones) and the Blocks (free rows, then provisioned ones) allow.  The
// first min(inserted, F) new keys take free rows.  The published count
// bounds both the IDMap occupancy and the rows allocated.
__device__ inline void reserve_rows(int64_t* cscal, int64_t* tscal, int64_t req, int64_t hw, int64_t keys, int64_t F,
                                    int64_t* h_live, int64_t tag) {
  const int64_t tombs = tscal[kTTomb];
  const int64_t key_room = max(tscal[kTLimit] - keys - tombs, int64_t(0));
  const int64_t row_room = F + max(tscal[kTRowCap] - hw, int64_t(0));
  const int64_t ins = min(req, min(key_room, row_room));
  const int64_t take = min(ins, F);
  cscal[kCNew] = ins;
  cscal[kCBaseLive] = hw;
  cscal[kCBaseKeys] = keys;
  cscal[kCFreeTop] = F;
  cscal[kCFreeTake] = take;
  cscal[kCTrunc] = req > ins ? 1 : 0;
  tscal[kTLive] = hw + ins - take;
  tscal[kTKeys] = keys + ins;
  tscal[kTFree] = F - take;
  publish_live(h_live, tag, max(keys + ins + tombs, hw + ins - take));
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
  if (nch == 1) {
    // one chunk: its totals are the totals (no chunk scan, no counter)
    if (threadIdx.x < 5) csum[threadIdx.x] = 0;
  } else {
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
  }
  if (threadIdx.x != 0) return;
  cscal[kCScanDone] = 0;  // ready for the next call on this workspace
  cscal[kCU] = tot[0];
  cscal[kCValid] = tot[1];
  cscal[kCNewReq] = tot[2];
  cscal[kCNLong] = tot[3];
  cscal[kCNUnits] = tot[4];
  reserve_rows(cscal, tscal, tot[2], tscal[kTLive], tscal[kTKeys], tscal[kTFree], h_live, tag);
}

// After the host grew the table: reserve again from the same counts.
__global__ void k_rereserve(int64_t* cscal, int64_t* tscal, int64_t* h_live, int64_t tag) {
  reserve_rows(cscal, tscal, cscal[kCNewReq], cscal[kCBaseLive], cscal[kCBaseKeys], cscal[kCFreeTop], h_live, tag);
}

__global__ void k_zero_scalars(int64_t* cscal) { cscal[threadIdx.x] = 0; }

hipError_t launch_rereserve(const Work& w, const TableDev& t, int64_t* h_live, int64_t tag, hipStream_t s) {
  k_rereserve<<<1, 1, 0, s>>>(w.scal, t.scal, h_live, tag);
  return hipGetLastError();
}

FrontGeom front_geom(int64_t n) {
  FrontGeom g;
  const int64_t n1 = n > 0 ? n : 1;
  g.ntiles = (n1 + kDedupTile - 1) / kDedupTile;
  g.R = std::min<int64_t>(kMaxTilesPerBlock, (g.ntiles + 255) / 256);
  g.nblk = (g.ntiles + g.R - 1) / g.R;
  g.rcap = g.R * kDedupTile;
  g.P = 1;
  g.logP = 0;
  // about 4096 ids (some 1500-2000 records) per partition: the partitions of
  // a batch up to ~3M ids are all resident at once (3 blocks per CU)
  while (g.P < kMaxParts && static_cast<int64_t>(g.P) * 4096 < n1) {
    g.P <<= 1;
    ++g.logP;
  }
  return g;
}

hipError_t launch_dedup_keys(const int64_t* values, int64_t n, const TableDev& t, const Work& w, hipEvent_t* ev_tile,
                             hipEvent_t* ev_part, hipStream_t s) {
  const FrontGeom& g = w.g;
  if (n <= 0 || g.nblk > kMaxDedupBlocks) return hipErrorInvalidValue;
  if (ev_tile && ev_tile[0]) (void)hipEventRecord(ev_tile[0], s);
  k_tile_dedup<kDedupThreads><<<static_cast<unsigned>(g.nblk), kDedupThreads, 0, s>>>(
      values, n, w, reinterpret_cast<int*>(t.scal + kTErr));
  if (ev_tile && ev_tile[1]) (void)hipEventRecord(ev_tile[1], s);
  if (ev_part && ev_part[0]) (void)hipEventRecord(ev_part[0], s);
  k_part_dedup<<<static_cast<unsigned>(g.P), kPartThreads, 0, s>>>(t, w, n);
  return hipGetLastError();
}

hipError_t launch_dedup_probe(const int64_t* values, int64_t n, const TableDev& t, const Work& w, int64_t* h_live,
                              int64_t tag, hipEvent_t* ev_tile, hipEvent_t* ev_part, hipStream_t s) {
  if (n <= 0) {
    k_zero_scalars<<<1, kCScalars, 0, s>>>(w.scal);
    return hipGetLastError();
  }
  const hipError_t e = launch_dedup_keys(values, n, t, w, ev_tile, ev_part, s);
  if (e != hipSuccess) return e;
  const int64_t nb = record_tiles(w.g);
  k_first_sums<kBlock><<<static_cast<unsigned>(nb), kBlock, 0, s>>>(w);
  const int64_t nch = (nb + kScanChunk - 1) / kScanChunk;
  k_scan5<kScanChunk / 1024><<<static_cast<unsigned>(nch), 1024, 0, s>>>(w.bsum, nb, w.ntiles, w.csum, nch, w.scal,
                                                                          t.scal, h_live, tag);
  if (ev_part && ev_part[1]) (void)hipEventRecord(ev_part[1], s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pass 7: unique ids, segments, rows, IDMap inserts
// ---------------------------------------------------------------------------

template <int NT>
__global__ __launch_bounds__(NT) void k_compact(TableDev t, Work w) {
  __shared__ int sh[NT / kWave + 1][5];
  const int b = blockIdx.x;
  if (blockIdx.x == 0 && threadIdx.x == 0 && w.scal[kCTrunc]) atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrFull);
  if (empty_record_tile(w, b)) return;  // block-uniform: no keys, nothing to write
  int pre[5];  // the record tile's exclusive prefixes (keys, count, new, hot, units)
  const int64_t nch = (static_cast<int64_t>(gridDim.x) + kScanChunk - 1) / kScanChunk;
#pragma unroll
  for (int a = 0; a < 5; ++a) pre[a] = w.bsum[a * w.ntiles + b] + w.csum[a * nch + b / kScanChunk];
  int f[4];
  first_records(w, b, f);
  KeyInfo ki[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) ki[k] = key_info(w, f[k]);  // all four reads in flight together
  int cf = 0, cc = 0, cn = 0, cl = 0, cu = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (f[k] < 0) continue;
    cf += 1;
    cc += ki[k].count;
    cn += ki[k].row < 0;
    if (ki[k].count > kLong) {
      cl += 1;
      cu += unit_count(ki[k].count);
    }
  }
  // the tile's keys get consecutive unique ids, segments, rows of new keys,
  // hot-key indices and backward units
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
  const int64_t ftop = w.scal[kCFreeTop], ftake = w.scal[kCFreeTake];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (f[k] < 0) continue;
    const int c = ki[k].count;
    const int64_t key = ki[k].key;
    w.unique[uid] = key;
    int li = -1;
    if (c > kLong) {
      li = lnext++;
      w.long_u[li] = uid;
      w.long_start[li] = unext;
      unext += unit_count(c);
    }
    int64_t row = ki[k].row;
    if (row < 0) {
      if (nr < inserted) {
        const int64_t slot = idmap_claim(t, static_cast<unsigned long long>(key) ^ kSign);
        if (slot >= 0) {
          // the first `ftake` new keys take free rows from the top of the stack
          row = nr < ftake ? t.free_rows[ftop - 1 - nr] : live0 + (nr - ftake);
          t.slots[slot].row = row;
          w.new_list[nr] = uid;
        } else {
          w.new_list[nr] = -1;  // no slot (cannot happen below the key limit): no row to initialise
          atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
        }
      }
      ++nr;
    } else if (t.meta_off >= 0) {
      // eviction: this call is the key's last lookup
      *reinterpret_cast<uint32_t*>(t.store.row(row) + t.meta_off + 8) = t.clock;
    }
    w.rows[uid] = row;
    w.useg[uid] = Seg{row, start, c};
    KeyInfo o = ki[k];
    o.row = row;
    o.uid = uid;
    o.start = start;
    o.long_idx = li;
    w.kinfo[f[k]] = o;
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
// formula, optimizer state zero, and for eviction the key and this call's
// clock; 16 bytes per lane per store.  Block `blk` of `nblk` takes every
// nblk-th group of keys.
__device__ inline void init_rows(const TableDev& t, const Work& w, int64_t blk, int64_t nblk) {
  constexpr int G = 16;
  const int lane = threadIdx.x % G, grp = threadIdx.x / G;
  const int64_t inserted = w.scal[kCNew];
  const int chunks = static_cast<int>(t.store.stride / 16);
  const int wbytes = t.dim * (t.row_dtype ? 2 : 4);
  for (int64_t q = blk * (kBlock / G) + grp; q < inserted; q += nblk * (kBlock / G)) {
    const int u = w.new_list[q];
    if (u < 0) continue;
    const int64_t row = w.useg[u].row;
    const int64_t key = w.unique[u];
    const uint64_t z = mix64(static_cast<uint64_t>(key) ^ mix64(t.seed));
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
      if (t.meta_off >= 0 && off + 16 > t.meta_off && off < t.meta_off + 12) {
        uint32_t v4[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int b = off + 4 * q4 - t.meta_off;  // byte of the {key, clock} record
          if (b == 0) v4[q4] = static_cast<uint32_t>(static_cast<uint64_t>(key));
          if (b == 4) v4[q4] = static_cast<uint32_t>(static_cast<uint64_t>(key) >> 32);
          if (b == 8) v4[q4] = t.clock;
        }
        val = make_uint4(v4[0], v4[1], v4[2], v4[3]);
      }
      *reinterpret_cast<uint4*>(rp + off) = val;
    }
  }
}

// The per-occurrence pass: inverse[i] = unique id of occurrence i (-1 for a
// rejected key).  For a forward (OCC) it also writes each occurrence's row
// and its position in the occurrence list (the key's segment start + the
// record's rank base + the rank inside the tile), and the descriptor of
// every backward unit of a hot key.
template <bool OCC>
__device__ inline void occ_pass(const Work& w, int64_t n, int64_t blk) {
  const int64_t i0 = (blk * kBlock + threadIdx.x) * 4;
  if (i0 >= n) return;
  const FrontGeom g = w.g;
  int ow[4];
  load4(reinterpret_cast<const int32_t*>(w.occ_word), i0, n, ow);  // -1 = kOccRejected past n
  int2 rr[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t o = static_cast<uint32_t>(ow[k]);
    const int64_t src = o == kOccRejected ? 0 : ((i0 + k) >> kDedupTileLog2) / g.R * g.rcap + (o >> 12);
    rr[k] = w.recres[src];  // all in flight together
  }
  KeyInfo a[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) a[k] = key_info(w, rr[k].x);
  int pos[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t o = static_cast<uint32_t>(ow[k]);
    if (o == kOccRejected) {
      a[k].row = -1;
      a[k].uid = -1;
      pos[k] = -1;
      continue;
    }
    const int rk = static_cast<int>(static_cast<uint32_t>(rr[k].y) & ~kRecFirst) + static_cast<int>(o & 0xFFFu);
    pos[k] = a[k].start + rk;
    if (OCC && a[k].long_idx >= 0) {
      const int sh = unit_shift(a[k].count);
      const int usz = kUnit << sh;
      if ((rk & (usz - 1)) == 0)
        w.units[w.long_start[a[k].long_idx] + (rk >> (kUnitLog2 + sh))] =
            Unit{a[k].long_idx, pos[k], min(pos[k] + usz, a[k].start + a[k].count), 0};
    }
  }
  if (i0 + 4 <= n) {
    // the inverse (the caller's) and the list positions (the backward's)
    // are not read in the forward: non-temporal
    store4_nt(w.inverse + i0, a[0].uid, a[1].uid, a[2].uid, a[3].uid);
    if (OCC) {
      *reinterpret_cast<longlong2*>(w.occ_row + i0) = make_longlong2(a[0].row, a[1].row);
      *reinterpret_cast<longlong2*>(w.occ_row + i0 + 2) = make_longlong2(a[2].row, a[3].row);
      store4_nt(w.occ_pos + i0, pos[0], pos[1], pos[2], pos[3]);
    }
  } else {
    for (int k = 0; k < 4 && i0 + k < n; ++k) {
      w.inverse[i0 + k] = a[k].uid;
      if (OCC) {
        w.occ_row[i0 + k] = a[k].row;
        w.occ_pos[i0 + k] = pos[k];
      }
    }
  }
}

// The last pass of a lookup: blocks [0, occ_blocks) run the per-occurrence
// pass, the others write the rows of the inserted keys (both only need the
// compaction, so they share one launch).
template <bool OCC>
__global__ __launch_bounds__(kBlock) void k_occ_init(TableDev t, Work w, int64_t n, int64_t occ_blocks) {
  const int64_t b = blockIdx.x;
  if (b < occ_blocks) occ_pass<OCC>(w, n, b);
  else init_rows(t, w, b - occ_blocks, static_cast<int64_t>(gridDim.x) - occ_blocks);
}

hipError_t launch_compact_insert(const int64_t* values, int64_t n, const TableDev& t, const Work& w, bool occ_lists,
                                 hipEvent_t* ev_compact, hipEvent_t* ev_init, hipEvent_t* ev_occ, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = record_tiles(w.g);
  if (ev_compact && ev_compact[0]) (void)hipEventRecord(ev_compact[0], s);
  k_compact<kBlock><<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, w);
  if (ev_compact && ev_compact[1]) (void)hipEventRecord(ev_compact[1], s);
  // one launch: the per-occurrence pass and the new rows (the init-rows and
  // occurrence events both bracket it)
  if (ev_init && ev_init[0]) (void)hipEventRecord(ev_init[0], s);
  if (ev_occ && ev_occ[0]) (void)hipEventRecord(ev_occ[0], s);
  const int64_t ob = grid_for(n, kBlock * 4, 1ll << 31);
  const int64_t ib = grid_for(n, kBlock / 16, 8192);
  if (occ_lists) k_occ_init<true><<<static_cast<unsigned>(ob + ib), kBlock, 0, s>>>(t, w, n, ob);
  else k_occ_init<false><<<static_cast<unsigned>(ob + ib), kBlock, 0, s>>>(t, w, n, ob);
  if (ev_occ && ev_occ[1]) (void)hipEventRecord(ev_occ[1], s);
  if (ev_init && ev_init[1]) (void)hipEventRecord(ev_init[1], s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// eviction of stale keys
// ---------------------------------------------------------------------------

// Slot index of an encoded key, or -1.
__device__ inline int64_t idmap_slot_of(const TableDev& t, unsigned long long e) {
  uint64_t h = idmap_hash(e) & t.cap_mask;
  for (uint64_t probed = 0; probed <= t.cap_mask; ++probed) {
    const unsigned long long k = t.slots[h].key;
    if (k == e) return static_cast<int64_t>(h);
    if (k == kEncEmpty) return -1;
    h = (h + 1) & t.cap_mask;
  }
  return -1;
}

// Row r holds a key whose age (clock - clock of its last lookup, mod 2^32)
// exceeds max_age.  Rows at or past the high-water mark hold nothing.
__device__ inline bool stale_row(const TableDev& t, int64_t r, int64_t hw, uint32_t max_age, int64_t& key) {
  key = INT64_MIN;
  if (r >= hw) return false;
  const uint8_t* m = t.store.row(r) + t.meta_off;
  key = *reinterpret_cast<const int64_t*>(m);
  const uint32_t seen = *reinterpret_cast<const uint32_t*>(m + 8);
  return key != INT64_MIN && static_cast<uint32_t>(t.clock - seen) > max_age;
}

// Stale rows per block of kEvictRows rows (4 per thread).
__global__ __launch_bounds__(kBlock) void k_evict_count(TableDev t, uint32_t max_age, int32_t* __restrict__ bcount) {
  __shared__ int sh[kBlock / kWave + 1];
  const int64_t hw = t.scal[kTLive];
  int c = 0;
#pragma unroll
  for (int k = 0; k < kEvictRows / kBlock; ++k) {
    int64_t key;
    c += stale_row(t, static_cast<int64_t>(blockIdx.x) * kEvictRows + k * kBlock + threadIdx.x, hw, max_age, key);
  }
  const int tot = block_sum<kBlock>(c, sh);
  if (threadIdx.x == 0) bcount[blockIdx.x] = tot;
}

// One block: exclusive scan of the nb block counts in place (chunks of 1024
// with a running carry); the total goes to bcount[nb].
__global__ __launch_bounds__(1024) void k_evict_scan(int32_t* __restrict__ bcount, int64_t nb) {
  __shared__ int sh[1024 / kWave + 1];
  int carry = 0;
  for (int64_t base = 0; base < nb; base += 1024) {
    const int64_t i = base + threadIdx.x;
    const int v = i < nb ? bcount[i] : 0;
    int tot;
    const int ex = block_excl_scan<1024>(v, sh, tot);
    if (i < nb) bcount[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) bcount[nb] = carry;
}

// The stale rows of a block, in row order: each is pushed on the free stack
// (after the rows already there), its key is cleared and its IDMap slot
// becomes a tombstone.
__global__ __launch_bounds__(kBlock) void k_evict_apply(TableDev t, uint32_t max_age,
                                                        const int32_t* __restrict__ bcount) {
  __shared__ int sh[kBlock / kWave + 1];
  constexpr int K = kEvictRows / kBlock;
  const int64_t hw = t.scal[kTLive];
  const int64_t F0 = t.scal[kTFree];
  // thread tid owns rows r0 + tid*K ... + K-1: row order = thread order
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kEvictRows + static_cast<int64_t>(threadIdx.x) * K;
  int64_t key[K];
  bool st[K];
  int c = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    st[k] = stale_row(t, r0 + k, hw, max_age, key[k]);
    c += st[k];
  }
  int tot;
  int pos = block_excl_scan<kBlock>(c, sh, tot);
  const int64_t base = F0 + bcount[blockIdx.x];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if (!st[k]) continue;
    t.free_rows[base + pos++] = r0 + k;
    *reinterpret_cast<int64_t*>(t.store.row(r0 + k) + t.meta_off) = INT64_MIN;
    const int64_t slot = idmap_slot_of(t, static_cast<unsigned long long>(key[k]) ^ kSign);
    if (slot >= 0) t.slots[slot].key = kEncTomb;
    else atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
  }
}

__global__ void k_evict_finish(int64_t* tscal, const int32_t* bcount, int64_t nb) {
  const int64_t n = bcount[nb];
  tscal[kTFree] += n;
  tscal[kTKeys] -= n;
  tscal[kTTomb] += n;
}

hipError_t launch_evict(const TableDev& t, int64_t rows_prov, uint32_t max_age, int32_t* bcount, hipStream_t s) {
  if (t.meta_off < 0) return hipErrorInvalidValue;
  const int64_t nb = std::max<int64_t>(1, (rows_prov + kEvictRows - 1) / kEvictRows);
  k_evict_count<<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, max_age, bcount);
  k_evict_scan<<<1, 1024, 0, s>>>(bcount, nb);
  k_evict_apply<<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, max_age, bcount);
  k_evict_finish<<<1, 1, 0, s>>>(t.scal, bcount, nb);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// compaction of the Blocks after eviction
// ---------------------------------------------------------------------------

// Row r holds a key (eviction writes INT64_MIN into a freed row's key field).
__device__ inline bool row_holds_key(const TableDev& t, int64_t r) {
  return *reinterpret_cast<const int64_t*>(t.store.row(r) + t.meta_off) != INT64_MIN;
}

// Per block of kEvictRows rows below the high-water mark hw: the free rows
// below the live count L ("holes") and the rows at or above L that hold a key
// ("movers").  Thread tid owns rows r0 + tid*K ... (row order = thread order).
__global__ __launch_bounds__(kBlock) void k_compact_count(TableDev t, int64_t L, int64_t hw, int32_t* __restrict__ hc,
                                                          int32_t* __restrict__ mc) {
  __shared__ int sh[kBlock / kWave + 1];
  constexpr int K = kEvictRows / kBlock;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kEvictRows + static_cast<int64_t>(threadIdx.x) * K;
  int h = 0, m = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int64_t r = r0 + k;
    if (r >= hw) continue;
    const bool held = row_holds_key(t, r);
    h += r < L && !held;
    m += r >= L && held;
  }
  const int th = block_sum<kBlock>(h, sh);
  __syncthreads();
  const int tm = block_sum<kBlock>(m, sh);
  if (threadIdx.x == 0) {
    hc[blockIdx.x] = th;
    mc[blockIdx.x] = tm;
  }
}

// The holes and the movers of each block, in row order, at their ranks
// (hc / mc hold the blocks' exclusive prefixes).
__global__ __launch_bounds__(kBlock) void k_compact_list(TableDev t, int64_t L, int64_t hw,
                                                         const int32_t* __restrict__ hc, const int32_t* __restrict__ mc,
                                                         int64_t* __restrict__ hole_at, int64_t* __restrict__ src_at,
                                                         int64_t cap) {
  __shared__ int sh[kBlock / kWave + 1];
  constexpr int K = kEvictRows / kBlock;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kEvictRows + static_cast<int64_t>(threadIdx.x) * K;
  bool hole[K], mover[K];
  int h = 0, m = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int64_t r = r0 + k;
    const bool held = r < hw && row_holds_key(t, r);
    hole[k] = r < hw && r < L && !held;
    mover[k] = r >= L && held;
    h += hole[k];
    m += mover[k];
  }
  int tot;
  int hp = hc[blockIdx.x] + block_excl_scan<kBlock>(h, sh, tot);
  int mp = mc[blockIdx.x] + block_excl_scan<kBlock>(m, sh, tot);
#pragma unroll
  for (int k = 0; k < K; ++k) {  // both lists hold at most cap = hw - L rows
    if (hole[k] && hp < cap) hole_at[hp] = r0 + k;
    if (mover[k] && mp < cap) src_at[mp] = r0 + k;
    hp += hole[k];
    mp += mover[k];
  }
}

// One wave per move: the k-th mover's row (values, state, key and clock)
// is copied into the k-th hole, 16 bytes per lane, and its IDMap slot takes
// the new row.  npairs: the device-side count (the movers' total).
__global__ __launch_bounds__(kBlock) void k_compact_move(TableDev t, const int64_t* __restrict__ hole_at,
                                                         const int64_t* __restrict__ src_at,
                                                         const int32_t* __restrict__ nholes,
                                                         const int32_t* __restrict__ nmovers, int64_t cap) {
  const int lane = threadIdx.x & (kWave - 1);
  // the two counts agree for a consistent table (both are the keys missing
  // below L); the minimum keeps every index inside the lists regardless
  const int64_t np = min(min(static_cast<int64_t>(*nholes), static_cast<int64_t>(*nmovers)), cap);
  if (blockIdx.x == 0 && threadIdx.x == 0 && *nholes != *nmovers)
    atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
  const int words = static_cast<int>(t.store.stride / 16);
  for (int64_t k = static_cast<int64_t>(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave; k < np;
       k += static_cast<int64_t>(gridDim.x) * (kBlock / kWave)) {
    const int64_t src = src_at[k], dst = hole_at[k];
    const uint4* sp = reinterpret_cast<const uint4*>(t.store.row(src));
    uint4* dp = reinterpret_cast<uint4*>(t.store.row(dst));
    for (int q = lane; q < words; q += kWave) dp[q] = sp[q];
    if (lane == 0) {
      const int64_t key = *reinterpret_cast<const int64_t*>(t.store.row(src) + t.meta_off);
      const int64_t slot = idmap_slot_of(t, static_cast<unsigned long long>(key) ^ kSign);
      if (slot >= 0) t.slots[slot].row = dst;
      else atomicOr(reinterpret_cast<int*>(&t.scal[kTErr]), kErrProbe);
    }
  }
}

__global__ void k_compact_finish(int64_t* tscal, int64_t L) {
  tscal[kTLive] = L;
  tscal[kTFree] = 0;
}

hipError_t launch_compact_rows(const TableDev& t, int64_t L, int64_t hw, int32_t* hc, int32_t* mc, int64_t* hole_at,
                               int64_t* src_at, hipStream_t s) {
  if (t.meta_off < 0 || hw <= L) return hipErrorInvalidValue;
  const int64_t nb = (hw + kEvictRows - 1) / kEvictRows;
  k_compact_count<<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, L, hw, hc, mc);
  k_evict_scan<<<1, 1024, 0, s>>>(hc, nb);  // exclusive prefixes; the totals at [nb]
  k_evict_scan<<<1, 1024, 0, s>>>(mc, nb);
  k_compact_list<<<static_cast<unsigned>(nb), kBlock, 0, s>>>(t, L, hw, hc, mc, hole_at, src_at, hw - L);
  k_compact_move<<<grid_for(hw - L, kBlock / kWave, 8192), kBlock, 0, s>>>(t, hole_at, src_at, hc + nb, mc + nb,
                                                                           hw - L);
  k_compact_finish<<<1, 1, 0, s>>>(t.scal, L);
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
      // state_elems floats per row ([s0 | s1 | row scalar], as present); the
      // thread of element j copies state floats j, j + dim, ...
      const int se = t.nstate * t.dim + t.rowscalar;
      const float* sp = ok ? reinterpret_cast<const float*>(rp + static_cast<int64_t>(t.dim) * (t.row_dtype ? 2 : 4)) : nullptr;
      for (int q = j; q < se; q += t.dim) state_out[i * se + q] = ok ? sp[q] : __builtin_nanf("");
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

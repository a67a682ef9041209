// Internal declarations shared by the kernels and the C ABI host code.
// gfx950 / CDNA4 only: 64-lane wavefronts, 256-thread blocks, 16-byte vector
// memory operations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "recis_mi355x.h"

namespace rs {

constexpr int kBlock = 256;  // threads per block (4 waves)
constexpr int kWave = 64;
constexpr uint64_t kSign = 0x8000000000000000ull;

// Stored keys are key ^ INT64_MIN, so the reserved keys INT64_MIN (empty)
// and INT64_MIN+1 (tombstone) become 0 and 1 and a zero-filled array is an
// empty table.
constexpr unsigned long long kEncEmpty = 0ull;
constexpr unsigned long long kEncTomb = 1ull;

// Dedup, pass 1: a block dedups tiles of kDedupTile occurrences in LDS
// (1024 threads x 4 occurrences, 8192 LDS hash slots) and writes one record
// per distinct key of a tile, with the key's hash partition.
constexpr int kDedupItems = 4;
constexpr int kDedupThreads = 1024;
constexpr int kDedupTile = kDedupThreads * kDedupItems;  // 4096
constexpr int kDedupTileLog2 = 12;
static_assert(kDedupTile == 1 << kDedupTileLog2, "tile is a power of two");
// A dedup block takes at most kMaxTilesPerBlock consecutive tiles, so a
// record index inside a block fits 19 bits (occ_word = index << 12 | rank),
// and there are at most kMaxDedupBlocks dedup blocks (n <= 2^28).
constexpr int kMaxTilesPerBlock = 128;
constexpr int kMaxDedupBlocks = 512;
// Hash partitions of the records (a power of two); one block per partition
// dedups its records in an LDS table of kPartSlots slots.  A partition of at
// most kPartThreads * kPartFast records is processed with every record of a
// thread in registers (unless its distinct keys overflow the table); a larger
// one in sweeps of at most kPartSweep records (a key's records share a
// sweep).
constexpr int kMaxParts = 4096;
constexpr int kPartThreads = 256;
constexpr int kPartSlots = 2048;
// Records per thread of the register pass: partitions a little above
// kPartSlots records (whose distinct keys still fit the table) stay there.
constexpr int kPartFast = 10;
constexpr int kPartSweep = kPartSlots * 3 / 4;       // LDS load <= 0.75

// Tile of the passes over positions (4 consecutive items per thread: many
// resident waves for these latency-bound passes).
constexpr int kRankItems = 4;
constexpr int kRankTile = kBlock * kRankItems;  // 1024
// Tiles per block of the tile-sum scan.
constexpr int kScanChunk = 2048;

// Open addressing with linear probing; a lookup reads kProbeBatch
// consecutive IDMap slots (64 bytes) per round trip.
constexpr int kProbeBatch = 4;

// Backward: a key with at most kLong occurrences is reduced by one lane
// group; a longer ("hot") key is cut into units of kUnit positions, each
// writing a partial sum row that one block per key then adds up.
constexpr int kLong = 32;
constexpr int kShortKeys = 2;  // short keys a lane group reduces together (fp32 gradients)
constexpr int kUnit = 32;
constexpr int kUnitLog2 = 5;
static_assert(kUnit == 1 << kUnitLog2, "kUnit is a power of two");
// A key with more than kUnit * kMaxUnits occurrences gets units of
// kUnit << shift positions, so no key has more than kMaxUnits partial rows.
constexpr int kMaxUnits = 1024;
__host__ __device__ inline int unit_shift(int count) {
  int sh = 0;
  while ((count - 1) >> (sh + kUnitLog2) >= kMaxUnits) ++sh;
  return sh;
}
__host__ __device__ inline int unit_count(int count) {
  const int usz = kUnit << unit_shift(count);
  return (count + usz - 1) / usz;
}

// Grid of the grid-stride kernels that loop over a device-side count: 8
// blocks of 256 threads per CU on 256 CUs.
constexpr int kResident = 2048;

// Latched device error bits.
enum : int { kErrKey = 1, kErrFull = 2, kErrProbe = 8 };

// Table-resident device scalars: rows ever allocated (the high-water mark),
// the IDMap key limit, rows provisioned, error bits, export counter, and for
// eviction the free-row stack size, live keys and IDMap tombstones (without
// eviction live keys = rows and the other two stay 0).
enum : int {
  kTLive = 0,
  kTLimit = 1,
  kTRowCap = 2,
  kTErr = 3,
  kTExport = 4,
  kTFree = 5,
  kTKeys = 6,
  kTTomb = 7,
  kTScalars = 8
};
// Per-call (context) device scalars.
enum : int {
  kCU = 0,         // unique keys
  kCNew = 1,       // keys inserted
  kCValid = 2,     // occurrences kept (= sum of per-key counts)
  kCBaseLive = 3,  // live rows before the insert
  kCNewReq = 4,    // keys not found (inserted if room)
  kCNLong = 5,     // keys with more than kLong occurrences
  kCNUnits = 6,    // backward units of those keys
  kCTrunc = 7,     // 1 if some keys not found had no room (latched as RS_EFULL)
  kCScanDone = 8,  // blocks of the tile-sum scan that have finished
  kCBaseKeys = 9,  // live keys before the insert
  kCFreeTop = 10,  // free-row stack size before the insert
  kCFreeTake = 11, // inserted keys that take a free row (the first ones)
  kCIdLo = 12,     // ids [lo, hi) lie in the pooled bags: offsets[0], offsets[bags]
  kCIdHi = 13,     //   clamped to [0, n] (written by the pool)
  kCScalars = 14
};

// Ids partition: at most kMaxShards owner shards.  Its device scalars: the
// dedup passes' error bits at kTErr (the slots of a table's scalars), then the
// scan's completion counter and the number of distinct keys.
constexpr int kMaxShards = 1024;
enum : int { kPCounter = kTScalars, kPTotal = kTScalars + 1, kPScalars = kTScalars + 2 };

// Blocking of the ids partition's owner passes (a pure function of n, G).
struct OwnerGeom {
  int64_t ch;     // rank tiles (kRankTile positions) per block, a power of two
  int64_t nb;     // blocks
  int64_t len;    // G * nb per-(shard, block) counts
  int64_t nch;    // scan chunks of the counts (<= kScanChunk)
  int nbits;      // bits of an owner index
  uint32_t gmask; // G - 1 if G is a power of two, else 0
};

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Hashes of the IDMap buckets and of the dedup partitions (different salts).
__device__ inline uint64_t idmap_hash(unsigned long long e) { return mix64(e ^ 0x2545F4914F6CDD1Dull); }
__device__ inline uint64_t part_hash(unsigned long long e) { return mix64(e ^ 0x5BD1E9955BD1E995ull); }

struct alignas(16) Slot {
  unsigned long long key;  // encoded key
  long long row;
};

// Blocks: chunks of 2^shift rows that never move.  By default they are
// physical chunks mapped back to back into one reserved virtual range, so
// row r is at base + r * stride; a table whose memory comes from a caller's
// allocator keeps a device table of chunk pointers instead (row r is row
// r mod 2^shift of chunk r >> shift).  A row is [w: D x row dtype | state0:
// D x fp32 | state1: D x fp32 (Adam) | row scalar (row-wise optimizers) |
// {key, clock of its last lookup} (tables with eviction)], padded to 16 bytes.
struct RowStore {
  uint8_t* base;                   // the mapped range (null with a chunk table)
  uint8_t* const* chunks;          // the chunk table, or null
  int64_t stride;                  // bytes per row
  int shift;                       // log2 of the rows per chunk
  __device__ inline uint8_t* row(int64_t r) const {
    if (chunks) return chunks[r >> shift] + (r & ((int64_t(1) << shift) - 1)) * stride;
    return base + r * stride;
  }
};

struct TableDev {
  Slot* slots;
  uint64_t cap_mask;  // slots - 1 (linear probing, slot granularity)
  RowStore store;
  int64_t* scal;  // kT* scalars
  int dim;
  int row_dtype;  // 0 f32, 1 bf16
  int nstate;     // per-element fp32 state vectors after w (0, 1 or 2)
  int rowscalar;  // 1: one fp32 state scalar per row follows them (row-wise optimizers)
  int meta_off;   // eviction: byte offset of the row's {int64 key, uint32 clock}; -1: none
  uint32_t clock; // eviction: the lookup clock of this call
  int64_t* free_rows;  // eviction: the free-row stack
  uint64_t seed;
  float lo, span;  // init: fma(u, span, lo)
};

// Geometry of the dedup passes for n occurrences (a pure function of n).
struct FrontGeom {
  int64_t ntiles;  // tiles of kDedupTile occurrences
  int64_t R;       // tiles per dedup block (<= kMaxTilesPerBlock)
  int64_t nblk;    // dedup blocks
  int64_t rcap;    // record capacity of one dedup block (R * kDedupTile)
  int P;           // hash partitions (power of two <= kMaxParts)
  int logP;
};

// Record of one distinct key of a dedup tile.  A tile's records are written
// in the order of the keys' first positions in the tile (so a block's
// records, tile after tile, are in first-position order), with meta = (rank
// of the record among its block's records of the same partition) << 12 |
// (count - 1); the block then copies its records into partition order with
// meta = (tile-order index) << 12 | (count - 1).
struct alignas(16) TileRec {
  unsigned long long key;  // encoded key
  unsigned int tmin;       // first position of the key in the tile
  unsigned int meta;
};

// One distinct key of the call, indexed by its key index: the tile-order
// position (in the record lists) of the key's first record.
struct alignas(32) KeyInfo {
  long long row;  // Blocks row (-1: not found / could not be inserted)
  long long key;  // the key
  int count;      // occurrences
  int uid;        // unique id (first-occurrence order)
  int start;      // first position of the key's segment of the occurrence list
  int long_idx;   // hot-key index, -1 if count <= kLong
};

// occ_word of a rejected (reserved) key
constexpr uint32_t kOccRejected = 0xFFFFFFFFu;

// Per-unique segment descriptor: the key's row, and where its occurrences
// start in the occurrence list and how many there are.
struct alignas(16) Seg {
  long long row;
  int start, count;
};

// Backward unit of a hot key: gradient-list positions [p0, p1), partial row li.
struct alignas(16) Unit {
  int li, p0, p1, pad;
};

// Workspace arrays of one forward (and its backward).
struct Work {
  uint32_t* occ_word;   // [n] dedup record index (in its block) << 12 | rank in the tile
  TileRec* trec;        // [nblk * rcap] records of the dedup tiles, per block, tile order
  int2* recres;         // [nblk * rcap] (same memory as trec) {key index, rank base | kRecFirst} per record
  int32_t* nrec;        // [nblk] records of each dedup block
  TileRec* srec;        // [nblk * rcap] the same records per block in partition order
  int32_t* pcnt;        // [nblk * P] records per (block, partition)
  int32_t* poff;        // [nblk * P] their offsets in the block's partition-ordered copy
  int2* ptmp;           // [nblk * rcap] per partition-ordered record: (tile-order index << 12 | LDS slot), rank base
  KeyInfo* kinfo;       // [nblk * rcap] per key index
  int64_t nkeyidx;      // nblk * rcap (key indices are below it)
  int32_t* inverse;     // [n]
  int64_t* occ_row;     // [n] Blocks row of each occurrence (-1: none)
  int32_t* occ_pos;     // [n] position of each occurrence in the occurrence list
  int64_t* unique;      // [n]
  Seg* useg;            // [n]
  int64_t* rows;        // [n]
  int32_t* new_list;    // [n] unique id of the k-th inserted key
  int32_t* id_ref;      // [n] gradient row of each id (written by the pool; -1: none)
  int32_t* occ_ref;     // [n] gradient row of each position of the occurrence list
  const int64_t* offsets;  // the forward's bag offsets (mean pooling: the backward's 1 / bag length)
  int32_t* long_u;      // [n/kLong + 1] unique id of each hot key
  int32_t* long_start;  // [n/kLong + 1] first backward unit of each hot key
  Unit* units;          // [2n/kUnit + 2] backward units of the hot keys
  int32_t* bsum;        // [5 * ntiles] record-tile sums: keys, their counts, new keys, hot keys, units
  int32_t* csum;        // [5 * (ntiles / kScanChunk + 1)] the same per chunk of record tiles
  int64_t* scal;        // [kCScalars]
  float* gpart;         // [(2n/kUnit + 2) * D] partial gradient row of each backward unit
  int64_t ntiles;       // record tiles (kRankTile records of one dedup block each; bsum stride)
  FrontGeom g;
};

// The record result of a key's first record (the one holding its first
// position) carries this bit in its rank-base word.
constexpr uint32_t kRecFirst = 0x80000000u;
// Record tiles: dedup block b's record slots [c * kRankTile, (c + 1) *
// kRankTile) for c < rcap / kRankTile, in block-major order.
inline int64_t record_tiles(const FrontGeom& g) { return g.nblk * (g.rcap / kRankTile); }

struct OptArgs {
  int opt;  // 0 adagrad, 1 adam, 2 adamw, 3 adam (epsilon-hat form), 4 row-wise adagrad, 5 row-wise adam
  float lr, eps, beta1, beta2, omb1, omb2, bc1, bc2;  // omb = 1 - beta, all derived in double
  float wdlr;  // lr * weight_decay (adamw)
  float lrt;   // lr * sqrt(1 - beta2^t) / (1 - beta1^t) (epsilon-hat form)
};

// Record `msg` as the calling thread's last error (rs_last_error) and return st.
rs_status set_last_error(rs_status st, const char* msg);

// ---------------------------------------------------------------------------
// launchers; all enqueue on `s` and return hipGetLastError()
// ---------------------------------------------------------------------------
// Geometry of the dedup passes for n occurrences.
FrontGeom front_geom(int64_t n);
// Dedup of the call's keys in first-occurrence order and the IDMap probe
// (ends before the insert): tile dedup, partition-count scan, scatter into
// partitions, per-partition dedup + probe, tile sums of the first
// occurrences and their scan.  The scan also stores (tag << 48) | (live rows
// after the call) to h_live (pinned host memory; may be null), so the host
// can refresh its bound on the live count without a copy or an event.
hipError_t launch_dedup_probe(const int64_t* values, int64_t n, const TableDev& t, const Work& w, int64_t* h_live,
                              int64_t tag, hipEvent_t* ev_tile, hipEvent_t* ev_part, hipStream_t s);
// The first two dedup passes only (tile dedup, per-partition dedup): each
// record's key index with the key's first record flagged and, unless
// w.kinfo is null, the key info of every distinct key (t.slots null: no
// IDMap probe, row 0).  With w.kinfo null a key index is the first record's
// position in the partition-ordered copies (whose entry there holds the
// key).  n > 0.
hipError_t launch_dedup_keys(const int64_t* values, int64_t n, const TableDev& t, const Work& w, hipEvent_t* ev_tile,
                             hipEvent_t* ev_part, hipStream_t s);
// Geometry of the ids partition's owner passes.
OwnerGeom owner_geom(int64_t n, int G);
// Ids partition of n ids into G shards: the dedup passes on w (no IDMap, no
// key info), owner counts (hist [og.len]), their scan (csum [og.nch]), the
// stable scatter of the distinct keys into keys_out and of their output
// slots into kslot [per key index], shard_offsets [G+1] and
// info [2] = {distinct keys, error bits}, then w.inverse [n].  pscal holds
// kPScalars scalars.
hipError_t launch_ids_partition(const int64_t* values, int64_t n, int G, uint64_t seed, const Work& w,
                                const OwnerGeom& og, int32_t* hist, int32_t* csum, int32_t* kslot, int64_t* pscal,
                                int64_t* keys_out, int64_t* shard_offsets, int64_t* info, hipStream_t s);
// unique / segments / rows / IDMap insert / row init, then the per-occurrence
// pass: inverse[] and, for a forward (occ_lists), each occurrence's row and
// list position and the hot keys' backward units
hipError_t launch_compact_insert(const int64_t* values, int64_t n, const TableDev& t, const Work& w, bool occ_lists,
                                 hipEvent_t* ev_compact, hipEvent_t* ev_init, hipEvent_t* ev_occ, hipStream_t s);
// redo the row reservation of the last scan after the table has grown
hipError_t launch_rereserve(const Work& w, const TableDev& t, int64_t* h_live, int64_t tag, hipStream_t s);
hipError_t launch_map_rows(const Work& w, int64_t n, int64_t* rows_out, int64_t* n_inserted, hipStream_t s);
hipError_t launch_find(const TableDev& t, const int64_t* keys, int64_t n, int64_t* rows_out, hipStream_t s);
hipError_t launch_pool(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags, int mode,
                       int64_t pad_len, void* out, uint8_t* mask, hipEvent_t* ev, hipStream_t s);
// Backward (+ optimizer when opt is set).  nref: rows of the upstream
// gradient (bags, or bags * pad_len for the padded modes); an occurrence-list
// entry outside [0, nref) -- left stale by offsets that do not cover every
// position -- contributes nothing instead of reading out of bounds.
hipError_t launch_bwd(const TableDev& t, const Work& w, int64_t nref, int64_t n, int mode,
                      const void* grad, float* grad_unique, const OptArgs* opt, hipEvent_t* ev_list,
                      hipEvent_t* ev_short, hipEvent_t* ev_long, hipStream_t s);
hipError_t launch_opt(const TableDev& t, const Work& w, int64_t n, const float* grad_unique, const OptArgs& opt,
                      hipEvent_t* ev, hipStream_t s);
// Feature transforms fused over ncols columns of one flat array of n
// elements (column c: [col_off[c], col_off[c+1])).
hipError_t launch_bucketize(const float* values, int64_t n, const int64_t* col_off, int ncols, const float* bnd,
                            const int64_t* bnd_off, int64_t* out, hipStream_t s);
hipError_t launch_mod(const int64_t* values, int64_t n, const int64_t* col_off, int ncols, const int64_t* moduli,
                      int64_t* out, hipStream_t s);
// Eviction of the keys whose age (clock - clock of their last lookup)
// exceeds max_age: their IDMap slots become tombstones and their rows are
// pushed on the free stack in row order.  bcount: one int per block of
// kEvictRows rows; the evicted count is added to the table scalars.
constexpr int kEvictRows = 1024;
hipError_t launch_evict(const TableDev& t, int64_t rows_prov, uint32_t max_age, int32_t* bcount, hipStream_t s);
// Bandwidth probes (measurement references).  read / write / copy: n bytes
// (a multiple of 16) of a (and b); gather / rmw: n random rows of row_bytes
// of a (a_bytes long) by idx, gathered into b or updated in place.
enum : int { kProbeRead = 0, kProbeWrite = 1, kProbeCopy = 2, kProbeGather = 3, kProbeRmw = 4 };
hipError_t launch_probe(int kind, void* a, int64_t a_bytes, void* b, const int64_t* idx, int64_t n, int row_bytes,
                        hipStream_t s);
// Lanes per row of the row probes for rows of w16 16-byte words (0: not supported).
int probe_lanes(int w16);
// Compaction after eviction: with L live keys and hw rows allocated, the
// k-th row at or above L holding a key moves (whole: values, state, key,
// clock) into the k-th free row below L, both in ascending order, and its
// IDMap slot follows; then hw = L and no row is free.  hc, mc: ints for
// ceil(hw / kEvictRows) + 1 blocks; hole_at, src_at: hw - L entries each.
hipError_t launch_compact_rows(const TableDev& t, int64_t L, int64_t hw, int32_t* hc, int32_t* mc, int64_t* hole_at,
                               int64_t* src_at, hipStream_t s);
hipError_t launch_rehash(const Slot* old_slots, int64_t old_cap, const TableDev& t, hipStream_t s);
hipError_t launch_export(const TableDev& t, int64_t cap_slots, int64_t* keys, int64_t* rows, int64_t cap,
                         int64_t* n_dev, hipStream_t s);
hipError_t launch_read_rows(const TableDev& t, const int64_t* rows, int64_t n, float* w_out, float* state_out,
                            hipStream_t s);

}  // namespace rs

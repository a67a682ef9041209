// Internal declarations shared by the kernels (kernels.hip) and the C ABI
// host code (api.hip).  gfx950 / CDNA4 only: 64-lane wavefronts, 256-thread
// blocks, 16-byte vector memory operations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rs {

constexpr int kBlock = 256;                  // threads per block (4 waves)
constexpr int kWave = 64;
constexpr uint64_t kSign = 0x8000000000000000ull;

// Stored keys are key ^ INT64_MIN, so the reserved keys INT64_MIN (empty)
// and INT64_MIN+1 (tombstone) become 0 and 1 and a zero-filled array is an
// empty table.
constexpr unsigned long long kEncEmpty = 0ull;
constexpr unsigned long long kEncTomb = 1ull;

// Dedup: a block dedups a tile of occurrences in LDS before touching the
// global scratch table, so a hot key costs one global atomic per tile.
constexpr int kDedupItems = 4;
constexpr int kDedupTile = kBlock * kDedupItems;  // 1024 occurrences
constexpr int kDedupLdsSlots = 2 * kDedupTile;    // load <= 0.5

// Block-tile scans: 8 consecutive items per thread.
constexpr int kScanItems = 8;
constexpr int kScanTile = kBlock * kScanItems;    // 2048

// Backward: the occurrence list (sorted by unique id) is cut into chunks of
// kChunk positions; a lane group reduces one chunk.
constexpr int kChunk = 32;

constexpr int kMaxBlocks = 1 << 16;               // Blocks chunks per table

// Latched device error bits.
enum : int { kErrKey = 1, kErrFull = 2, kErrScratch = 4, kErrProbe = 8 };

// Table-resident device scalars.
enum : int { kTLive = 0, kTLimit = 1, kTRowCap = 2, kTErr = 3, kTExport = 4, kTScalars = 8 };
// Per-call (context) device scalars.
enum : int { kCU = 0, kCNew = 1, kCValid = 2, kCBaseLive = 3, kCScalars = 4 };

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Slot hash of the IDMap and of the dedup scratch (different salts).
__device__ inline uint64_t idmap_hash(unsigned long long e) { return mix64(e ^ 0x2545F4914F6CDD1Dull); }
__device__ inline uint64_t scratch_hash(unsigned long long e) { return mix64(e ^ 0x5BD1E9955BD1E995ull); }

struct alignas(16) Slot {
  unsigned long long key;  // encoded key
  long long row;
};

// Blocks: rows live in fixed-size chunks that never move; a row is
// [w: D x row dtype | state0: D x fp32 | state1: D x fp32 (Adam)].
struct RowStore {
  uint8_t* const* blocks;  // device array of chunk base pointers
  int shift;               // log2(block_rows)
  int64_t mask;            // block_rows - 1
  int64_t stride;          // bytes per row
  __device__ inline uint8_t* row(int64_t r) const {
    return blocks[r >> shift] + (r & mask) * stride;
  }
};

struct TableDev {
  Slot* slots;
  uint64_t cap_mask;
  RowStore store;
  int64_t* scal;  // kT* scalars
  int dim;
  int row_dtype;  // 0 f32, 1 bf16
  int nstate;     // 1 or 2
  uint64_t seed;
  float lo, span;  // init: fma(u, span, lo)
};

struct Scratch {
  unsigned long long* key;
  unsigned int* first;
  unsigned int* cnt;
  int32_t* uid;
  uint64_t mask;
};

// Workspace arrays of one forward (and its backward).
struct Work {
  int32_t* slot_of;   // [n] scratch slot per occurrence
  int32_t* occ_rank;  // [n] rank of the occurrence among those of its key
  int32_t* inverse;   // [n]
  int64_t* unique;    // [n]
  int32_t* uslot;     // [n] scratch slot per unique
  int32_t* ucount;    // [n] occurrences per unique
  int32_t* seg;       // [n+1] exclusive scan of ucount
  int64_t* rows;      // [n]
  int32_t* isnew;     // [n]
  int32_t* occ_ref;   // [n] grad row of each position of the occurrence list
  int32_t* chunk_u;   // [n/kChunk + 1] unique id at the start of each chunk
  int32_t* bsum;      // [n/kScanTile + 2] tile sums
  int64_t* scal;      // [kCScalars]
  float* gpart;       // [(n/kChunk + 1) * D] partial sums of segments crossing chunks
};

struct OptArgs {
  int opt;  // 0 adagrad, 1 adam
  float lr, eps, beta1, beta2, omb1, omb2, bc1, bc2;  // omb = 1 - beta, all derived in double
};

// ---------------------------------------------------------------------------
// launchers (kernels.hip); all enqueue on `s` and return hipGetLastError()
// ---------------------------------------------------------------------------
hipError_t launch_fill_u64(unsigned long long* p, unsigned long long v, int64_t n, hipStream_t s);

hipError_t launch_dedup(const int64_t* values, int64_t n, const Scratch& sc, const Work& w,
                        int* err, hipEvent_t* ev_local, hipEvent_t* ev_compact, hipStream_t s);
hipError_t launch_seg_scan(const Work& w, int64_t nmax, const Scratch& sc, int dim, hipStream_t s);
hipError_t launch_idmap_probe(const TableDev& t, const Work& w, int64_t nmax, hipEvent_t* ev,
                              hipStream_t s);
hipError_t launch_idmap_insert(const TableDev& t, const Work& w, int64_t nmax, hipEvent_t* ev,
                               hipStream_t s);
hipError_t launch_map_rows(const Work& w, int64_t n, int64_t* rows_out, int64_t* n_inserted,
                           hipStream_t s);
hipError_t launch_find(const TableDev& t, const int64_t* keys, int64_t n, int64_t* rows_out,
                       hipStream_t s);
hipError_t launch_pool(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n, int64_t bags,
                       int mode, int64_t pad_len, void* out, uint8_t* mask, hipEvent_t* ev,
                       hipStream_t s);
hipError_t launch_bwd(const TableDev& t, const Work& w, const int64_t* offsets, int64_t n,
                      int64_t bags, int mode, int64_t pad_len, const void* grad, float* grad_unique,
                      const OptArgs* opt, hipEvent_t* ev_chunks, hipEvent_t* ev_straddle,
                      hipStream_t s);
hipError_t launch_opt(const TableDev& t, const Work& w, int64_t n, const float* grad_unique,
                      const OptArgs& opt, hipEvent_t* ev, hipStream_t s);
hipError_t launch_rehash(const Slot* old_slots, int64_t old_cap, const TableDev& t, hipStream_t s);
hipError_t launch_export(const TableDev& t, int64_t cap_slots, int64_t* keys, int64_t* rows,
                         int64_t cap, int64_t* n_dev, hipStream_t s);
hipError_t launch_read_rows(const TableDev& t, const int64_t* rows, int64_t n, float* w_out,
                            float* state_out, hipStream_t s);

}  // namespace rs

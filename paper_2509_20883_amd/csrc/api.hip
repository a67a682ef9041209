// C ABI of the sparse embedding step (declared in include/recis_mi355x.h).
//
// Host side of the two-tier store (RecIS, "Optimization for Memory Bound"):
// the IDMap is one open-addressing array of 16-byte slots {key, row} in HBM;
// the Blocks are fixed-size chunks of rows that are appended as the table
// grows and never move, so growing the IDMap only rehashes 16 bytes per key.
// The host never reads per-step sizes back unless the table may have to grow
// this step; it keeps an upper bound of the live row count instead.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "recis_mi355x.h"
#include "rs_internal.h"

using namespace rs;

static_assert(RS_PROBE_READ == kProbeRead && RS_PROBE_WRITE == kProbeWrite && RS_PROBE_COPY == kProbeCopy &&
                  RS_PROBE_GATHER == kProbeGather && RS_PROBE_RMW == kProbeRmw,
              "probe kinds of the header and the kernels agree");

namespace {

thread_local std::string g_last_error;

rs_status fail(rs_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

#define RS_HIP(call)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      return fail(RS_EHIP, std::string(#call) + ": " + hipGetErrorString(e_));                \
  } while (0)

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

bool padded_mode(int32_t mode) { return mode == RS_POOL_NONE || mode == RS_POOL_TILE_TAIL; }

// Workspace layout of one forward: every array sized by the upper bound n.
struct Layout {
  size_t occ_word, trec, nrec, srec, pcnt, poff, ptmp, kinfo, inverse, occ_row, occ_pos, unique, useg, rows,
      new_list, id_ref, occ_ref, long_u, long_start, units, bsum, csum, scal, gpart, total;
  int64_t ntiles;
  FrontGeom g;
};

Layout make_layout(int64_t n, int dim) {
  const size_t n1 = static_cast<size_t>(n > 0 ? n : 1);
  const size_t nlong = n1 / kLong + 1;        // keys with > kLong occurrences
  const size_t nunit = 2 * (n1 / kUnit) + 2;  // >= sum over them of ceil(count / kUnit)
  Layout L{};
  L.g = front_geom(n);
  L.ntiles = record_tiles(L.g);
  const size_t nrecs = static_cast<size_t>(L.g.nblk) * static_cast<size_t>(L.g.rcap);
  const size_t npc = static_cast<size_t>(L.g.P) * static_cast<size_t>(L.g.nblk);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.occ_word = take(4 * n1);
  L.trec = take(sizeof(TileRec) * nrecs);  // also the records' results (int2 each)
  L.nrec = take(4 * static_cast<size_t>(L.g.nblk));
  L.srec = take(sizeof(TileRec) * nrecs);
  L.pcnt = take(4 * npc);
  L.poff = take(4 * npc);
  L.ptmp = take(8 * nrecs);
  L.kinfo = take(sizeof(KeyInfo) * nrecs);
  L.inverse = take(4 * n1);
  L.occ_row = take(8 * n1);
  L.occ_pos = take(4 * n1);
  L.unique = take(8 * n1);
  L.useg = take(sizeof(Seg) * n1);
  L.rows = take(8 * n1);
  L.new_list = take(4 * n1);
  L.id_ref = take(4 * n1);
  L.occ_ref = take(4 * n1);
  L.long_u = take(4 * nlong);
  L.long_start = take(4 * nlong);
  L.units = take(sizeof(Unit) * nunit);
  L.bsum = take(4 * 5 * static_cast<size_t>(L.ntiles));
  L.csum = take(4 * 5 * static_cast<size_t>(L.ntiles / kScanChunk + 1));
  L.scal = take(8 * kCScalars);
  L.gpart = take(4 * nunit * static_cast<size_t>(dim));
  L.total = off;
  return L;
}

Work make_work(void* base, const Layout& L) {
  uint8_t* b = static_cast<uint8_t*>(base);
  Work w;
  w.occ_word = reinterpret_cast<uint32_t*>(b + L.occ_word);
  w.trec = reinterpret_cast<TileRec*>(b + L.trec);
  w.recres = reinterpret_cast<int2*>(b + L.trec);
  w.nrec = reinterpret_cast<int32_t*>(b + L.nrec);
  w.srec = reinterpret_cast<TileRec*>(b + L.srec);
  w.pcnt = reinterpret_cast<int32_t*>(b + L.pcnt);
  w.poff = reinterpret_cast<int32_t*>(b + L.poff);
  w.ptmp = reinterpret_cast<int2*>(b + L.ptmp);
  w.kinfo = reinterpret_cast<KeyInfo*>(b + L.kinfo);
  w.nkeyidx = L.g.nblk * L.g.rcap;
  w.inverse = reinterpret_cast<int32_t*>(b + L.inverse);
  w.occ_row = reinterpret_cast<int64_t*>(b + L.occ_row);
  w.occ_pos = reinterpret_cast<int32_t*>(b + L.occ_pos);
  w.unique = reinterpret_cast<int64_t*>(b + L.unique);
  w.useg = reinterpret_cast<Seg*>(b + L.useg);
  w.rows = reinterpret_cast<int64_t*>(b + L.rows);
  w.new_list = reinterpret_cast<int32_t*>(b + L.new_list);
  w.id_ref = reinterpret_cast<int32_t*>(b + L.id_ref);
  w.occ_ref = reinterpret_cast<int32_t*>(b + L.occ_ref);
  w.offsets = nullptr;
  w.long_u = reinterpret_cast<int32_t*>(b + L.long_u);
  w.long_start = reinterpret_cast<int32_t*>(b + L.long_start);
  w.units = reinterpret_cast<Unit*>(b + L.units);
  w.bsum = reinterpret_cast<int32_t*>(b + L.bsum);
  w.csum = reinterpret_cast<int32_t*>(b + L.csum);
  w.scal = reinterpret_cast<int64_t*>(b + L.scal);
  w.gpart = reinterpret_cast<float*>(b + L.gpart);
  w.ntiles = L.ntiles;
  w.g = L.g;
  return w;
}

// Workspace layout of one ids partition: the dedup passes' arrays (no
// IDMap), the owner counts and their scan, scalars.
struct PartLayout {
  size_t occ_word, trec, nrec, srec, pcnt, poff, ptmp, kslot, hist, csum, cscal, pscal, total;
  FrontGeom g;
  OwnerGeom og;
};

PartLayout make_part_layout(int64_t n, int G) {
  const size_t n1 = static_cast<size_t>(n > 0 ? n : 1);
  PartLayout L{};
  L.g = front_geom(n);
  L.og = owner_geom(record_tiles(L.g) * kRankTile, G);  // the owner passes walk the record slots
  const size_t nrecs = static_cast<size_t>(L.g.nblk) * static_cast<size_t>(L.g.rcap);
  const size_t npc = static_cast<size_t>(L.g.P) * static_cast<size_t>(L.g.nblk);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.occ_word = take(4 * n1);
  L.trec = take(sizeof(TileRec) * nrecs);
  L.nrec = take(4 * static_cast<size_t>(L.g.nblk));
  L.srec = take(sizeof(TileRec) * nrecs);
  L.pcnt = take(4 * npc);
  L.poff = take(4 * npc);
  L.ptmp = take(8 * nrecs);
  L.kslot = take(4 * nrecs);
  L.hist = take(4 * static_cast<size_t>(L.og.len));
  L.csum = take(4 * static_cast<size_t>(L.og.nch));
  L.cscal = take(8 * kCScalars);
  L.pscal = take(8 * kPScalars);
  L.total = off;
  return L;
}

Work make_part_work(void* base, const PartLayout& L, int32_t* inverse) {
  uint8_t* b = static_cast<uint8_t*>(base);
  Work w{};
  w.occ_word = reinterpret_cast<uint32_t*>(b + L.occ_word);
  w.trec = reinterpret_cast<TileRec*>(b + L.trec);
  w.recres = reinterpret_cast<int2*>(b + L.trec);
  w.nrec = reinterpret_cast<int32_t*>(b + L.nrec);
  w.srec = reinterpret_cast<TileRec*>(b + L.srec);
  w.pcnt = reinterpret_cast<int32_t*>(b + L.pcnt);
  w.poff = reinterpret_cast<int32_t*>(b + L.poff);
  w.ptmp = reinterpret_cast<int2*>(b + L.ptmp);
  w.kinfo = nullptr;  // no key info: only first-occurrence markers and key indices
  w.nkeyidx = L.g.nblk * L.g.rcap;
  w.inverse = inverse;
  w.scal = reinterpret_cast<int64_t*>(b + L.cscal);
  w.g = L.g;
  return w;
}

const char* err_text(int bits) {
  if (bits & kErrKey) return "a reserved key (INT64_MIN or INT64_MIN+1) was in the input";
  if (bits & kErrFull) return "the table is full (auto_grow is off): some keys were not inserted";
  if (bits & kErrProbe) return "IDMap probe found no free slot";
  return "device error";
}

rs_status err_status(int bits) {
  if (bits & kErrKey) return RS_EKEY;
  if (bits & kErrFull) return RS_EFULL;
  return RS_EHIP;
}

}  // namespace

rs_status rs::set_last_error(rs_status st, const char* msg) { return fail(st, msg); }

struct rs_table {
  rs_table_desc d{};
  rs_allocator a{};
  bool custom = false;
  int device = 0;
  // IDMap
  Slot* slots = nullptr;
  int64_t cap = 0;
  int64_t limit = 0;  // floor(max_load * cap)
  // Blocks: physical chunks (hipMemCreate) mapped back to back into one
  // reserved virtual range, so rows never move when the table grows
  uint8_t* va_base = nullptr;
  size_t va_size = 0;
  size_t mapped = 0;      // bytes mapped so far
  size_t chunk_bytes = 0; // block_rows * stride, rounded up to the mapping granularity
  std::vector<hipMemGenericAllocationHandle_t> chunks;
  // Blocks from the caller's allocator: one allocation per chunk of
  // block_rows rows, and a device table of their addresses
  std::vector<void*> achunks;
  uint8_t** d_chunk_tab = nullptr;
  int64_t chunk_tab_cap = 0;
  int64_t stride = 0;
  int64_t rows_prov = 0;
  // device scalars
  int64_t* d_scal = nullptr;
  // eviction: row metadata offset (-1: none), the lookup clock (one tick per
  // lookup call), the free-row stack (capacity rows_prov)
  int meta_off = -1;
  uint32_t clock = 0;
  int64_t* free_rows = nullptr;
  int64_t free_cap = 0;
  // host view of the live count: an upper bound.  Every insert call gets a
  // 16-bit tag; its scan kernel stores (tag << 48) | exact live count into
  // h_pin[0], and bound_after[tag % kTags] remembers the host's bound right
  // after that call was enqueued, so a published count refreshes the bound
  // by the calls enqueued since (bound_after[.] = -1: no refresh from it).
  static constexpr int kTags = 64;
  int64_t live_bound = 0;
  int64_t* h_pin = nullptr;
  int64_t tag = 0;
  int64_t bound_after[kTags];
  int64_t adam_t = 0;
  // internal workspace for ht_find_or_insert
  void* iws = nullptr;
  size_t iws_bytes = 0;
  hipEvent_t kev[RS_K_COUNT][2] = {};

  void* alloc(size_t bytes) {
    if (bytes == 0) bytes = 1;
    if (custom) return a.alloc(bytes, a.ctx);
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    return p;
  }
  void release(void* p) {
    if (!p) return;
    if (custom) a.free(p, a.ctx);
    else (void)hipFree(p);
  }
  // per-element state vectors, the row scalar of the row-wise optimizers
  int nstate() const {
    return d.optimizer == RS_ADAGRAD ? 1 : d.optimizer == RS_ADAGRAD_ROWWISE ? 0 : d.optimizer == RS_ADAM_ROWWISE ? 1 : 2;
  }
  int rowscalar() const { return d.optimizer == RS_ADAGRAD_ROWWISE || d.optimizer == RS_ADAM_ROWWISE ? 1 : 0; }
  int state_elems() const { return nstate() * d.dim + rowscalar(); }
  int wbytes() const { return d.row_dtype == RS_BF16 ? 2 : 4; }

  TableDev dev() const {
    TableDev t;
    t.slots = slots;
    t.cap_mask = static_cast<uint64_t>(cap - 1);
    t.store.base = va_base;
    t.store.chunks = d_chunk_tab;
    t.store.stride = stride;
    int sh = 0;
    while ((int64_t(1) << sh) < d.block_rows) ++sh;
    t.store.shift = sh;
    t.scal = d_scal;
    t.dim = d.dim;
    t.row_dtype = d.row_dtype;
    t.nstate = nstate();
    t.rowscalar = rowscalar();
    t.meta_off = meta_off;
    t.clock = clock;
    t.free_rows = free_rows;
    t.seed = d.seed;
    t.lo = d.init_lo;
    t.span = d.init_hi - d.init_lo;  // fp32 subtraction
    return t;
  }
  hipEvent_t* ev(int k) { return (kev[k][0] || kev[k][1]) ? kev[k] : nullptr; }
};

namespace {

__global__ void k_set_scalar(int64_t* p, int64_t v) { *p = v; }

rs_status set_scalar(rs_table* t, int idx, int64_t v, hipStream_t s) {
  k_set_scalar<<<1, 1, 0, s>>>(t->d_scal + idx, v);
  RS_HIP(hipGetLastError());
  return RS_OK;
}

rs_status take_latched(rs_table* t) {
  int64_t e = 0;
  RS_HIP(hipMemcpy(&e, t->d_scal + kTErr, sizeof(int64_t), hipMemcpyDeviceToHost));
  if (e == 0) return RS_OK;
  const int64_t zero = 0;
  RS_HIP(hipMemcpy(t->d_scal + kTErr, &zero, sizeof(int64_t), hipMemcpyHostToDevice));
  return fail(err_status(static_cast<int>(e)), err_text(static_cast<int>(e)));
}

// Add Blocks chunks from the caller's allocator until `rows` rows fit.
rs_status provision_alloc_rows(rs_table* t, int64_t rows, hipStream_t s) {
  while (t->rows_prov < rows) {
    const int64_t c = static_cast<int64_t>(t->achunks.size());
    if (c >= t->chunk_tab_cap) return fail(RS_ENOMEM, "table rows exceed the device's memory");
    void* p = t->alloc(t->chunk_bytes);
    if (!p) return fail(RS_ENOMEM, "the allocator returned NULL for a Blocks chunk");
    t->achunks.push_back(p);
    k_set_scalar<<<1, 1, 0, s>>>(reinterpret_cast<int64_t*>(t->d_chunk_tab) + c,
                                 static_cast<int64_t>(reinterpret_cast<uintptr_t>(p)));
    RS_HIP(hipGetLastError());
    t->rows_prov += t->d.block_rows;
  }
  return RS_OK;
}

// Map Blocks chunks until `rows` rows fit.
rs_status provision_rows(rs_table* t, int64_t rows, hipStream_t s) {
  if (rows <= t->rows_prov) return RS_OK;
  const size_t need = static_cast<size_t>(rows) * static_cast<size_t>(t->stride);
  if (t->custom) {
    rs_status st = provision_alloc_rows(t, rows, s);
    if (st != RS_OK) return st;
  } else if (need > t->va_size) {
    return fail(RS_ENOMEM, "table rows exceed the reserved Blocks address range");
  }
  hipMemAllocationProp prop = {};
  prop.type = hipMemAllocationTypePinned;
  prop.location.type = hipMemLocationTypeDevice;
  prop.location.id = t->device;
  hipMemAccessDesc acc = {};
  acc.location.type = hipMemLocationTypeDevice;
  acc.location.id = t->device;
  acc.flags = hipMemAccessFlagsProtReadWrite;
  while (!t->custom && t->mapped < need) {
    const size_t bytes = std::min(t->chunk_bytes, t->va_size - t->mapped);
    hipMemGenericAllocationHandle_t h;
    if (hipMemCreate(&h, bytes, &prop, 0) != hipSuccess) {
      (void)hipGetLastError();
      return fail(RS_ENOMEM, "hipMemCreate of a Blocks chunk failed");
    }
    if (hipMemMap(t->va_base + t->mapped, bytes, 0, h, 0) != hipSuccess ||
        hipMemSetAccess(t->va_base + t->mapped, bytes, &acc, 1) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipMemRelease(h);
      return fail(RS_EHIP, "mapping a Blocks chunk failed");
    }
    t->chunks.push_back(h);
    t->mapped += bytes;
  }
  if (!t->custom) t->rows_prov = static_cast<int64_t>(t->mapped / static_cast<size_t>(t->stride));
  if (t->meta_off >= 0 && t->rows_prov > t->free_cap) {
    // the free-row stack can hold every row
    int64_t* nf = static_cast<int64_t*>(t->alloc(sizeof(int64_t) * static_cast<size_t>(t->rows_prov)));
    if (!nf) return fail(RS_ENOMEM, "allocation of the free-row stack failed");
    if (t->free_rows) {
      RS_HIP(hipMemcpyAsync(nf, t->free_rows, sizeof(int64_t) * static_cast<size_t>(t->free_cap),
                            hipMemcpyDeviceToDevice, s));
      RS_HIP(hipStreamSynchronize(s));
      t->release(t->free_rows);
    }
    t->free_rows = nf;
    t->free_cap = t->rows_prov;
  }
  return set_scalar(t, kTRowCap, t->rows_prov, s);
}

// Rehash the IDMap into new_cap slots (stream-ordered; synchronizes).
rs_status rehash(rs_table* t, int64_t new_cap, hipStream_t s) {
  Slot* ns = static_cast<Slot*>(t->alloc(sizeof(Slot) * static_cast<size_t>(new_cap)));
  if (!ns) return fail(RS_ENOMEM, "allocation of the grown IDMap failed");
  RS_HIP(hipMemsetAsync(ns, 0, sizeof(Slot) * static_cast<size_t>(new_cap), s));
  Slot* old = t->slots;
  const int64_t old_cap = t->cap;
  t->slots = ns;
  t->cap = new_cap;
  t->limit = static_cast<int64_t>(std::floor(static_cast<double>(t->d.max_load) * static_cast<double>(new_cap)));
  RS_HIP(launch_rehash(old, old_cap, t->dev(), s));
  rs_status st = set_scalar(t, kTLimit, t->limit, s);
  if (st != RS_OK) return st;
  st = set_scalar(t, kTTomb, 0, s);  // the rehash leaves the tombstones behind
  if (st != RS_OK) return st;
  RS_HIP(hipStreamSynchronize(s));
  t->release(old);
  return RS_OK;
}

// Grow (when allowed) so that `keys_need` live keys fit the IDMap and
// `rows_need` rows the Blocks.  `batch` (the ids of the call) sizes the
// headroom: the IDMap is doubled until another call of `batch` ids would fit
// as well, so the host's upper bound on the live count (live + ids of the
// call) does not force a synchronization on every call of a batch larger
// than the free room.  Tombstones (eviction) count against the key limit
// until a rehash drops them: the IDMap is rehashed, at the same capacity if
// that suffices, when they would not leave that room.
rs_status grow_for(rs_table* t, int64_t keys_need, int64_t tombs, int64_t rows_need, int64_t batch, hipStream_t s) {
  if (t->d.auto_grow) {
    const double ml = static_cast<double>(t->d.max_load);
    int64_t c = t->cap;
    while (static_cast<double>(keys_need + batch) > ml * static_cast<double>(c)) c <<= 1;
    if (c != t->cap || static_cast<double>(keys_need + tombs + batch) > ml * static_cast<double>(c)) {
      rs_status st = rehash(t, c, s);
      if (st != RS_OK) return st;
    }
    // headroom: a quarter more rows and at least four batches' worth, so the
    // host's upper bound on live rows rarely forces a synchronization
    const int64_t headroom = rows_need + std::max(rows_need / 4, 4 * batch) + t->d.block_rows;
    return provision_rows(t, headroom, s);
  }
  return provision_rows(t, std::min(rows_need, t->limit), s);
}

// Lower the host's bound on live rows with the newest count a scan kernel
// has published (calls enqueued after it keep their share of the bound).
void refresh_bound(rs_table* t) {
  const int64_t v = __atomic_load_n(t->h_pin, __ATOMIC_ACQUIRE);
  const int64_t tag = (v >> 48) & 0xFFFF;
  if (tag == 0 || ((t->tag - tag) & 0xFFFF) >= rs_table::kTags) return;
  const int64_t after = t->bound_after[tag % rs_table::kTags];
  if (after < 0) return;
  const int64_t exact = v & ((int64_t(1) << 48) - 1);
  t->live_bound = std::min(t->live_bound, exact + (t->live_bound - after));
}

// The bound becomes exact (after a synchronization): counts published for
// earlier calls can no longer refresh it.
void reset_bound(rs_table* t, int64_t exact) {
  t->live_bound = exact;
  for (int64_t& b : t->bound_after) b = -1;
}

int64_t next_tag(rs_table* t) {
  t->tag = (t->tag & 0xFFFF) == 0xFFFF ? 1 : t->tag + 1;  // tags 1..65535 (0: nothing published)
  t->bound_after[t->tag % rs_table::kTags] = -1;
  return t->tag;
}

// Dedup `values` into w, then find-or-insert the unique keys (growing the
// table first when it may not have room).
rs_status dedup_and_insert(rs_table* t, const int64_t* values, int64_t n, const Work& w, bool occ_lists,
                           hipStream_t s) {
  rs_status st = RS_OK;
  const int64_t tag = next_tag(t);
  RS_HIP(launch_dedup_probe(values, n, t->dev(), w, t->h_pin, tag, t->ev(RS_K_TILE_DEDUP), t->ev(RS_K_PARTITION), s));
  refresh_bound(t);
  const int64_t bound = t->live_bound + n;
  if (bound > t->limit || bound > t->rows_prov) {
    // exact decision: read back U and live (one synchronization)
    RS_HIP(hipStreamSynchronize(s));
    // the scan already reserved rows for the keys not found (or as many as
    // fitted): read the request and the counts before it
    int64_t cs[kCScalars], ts[kTScalars];
    RS_HIP(hipMemcpy(cs, w.scal, sizeof(cs), hipMemcpyDeviceToHost));
    RS_HIP(hipMemcpy(ts, t->d_scal, sizeof(ts), hipMemcpyDeviceToHost));
    const int64_t req = cs[kCNewReq];
    const int64_t keys_need = cs[kCBaseKeys] + req;
    const int64_t rows_need = cs[kCBaseLive] + std::max<int64_t>(req - cs[kCFreeTop], 0);
    st = grow_for(t, keys_need, ts[kTTomb], rows_need, n, s);
    if (st != RS_OK) {
      // no memory to grow: undo the scan's row reservation, so the call
      // leaves the table as it found it (nothing inserted)
      const rs_status e1 = set_scalar(t, kTLive, cs[kCBaseLive], s);
      const rs_status e2 = set_scalar(t, kTKeys, cs[kCBaseKeys], s);
      const rs_status e3 = set_scalar(t, kTFree, cs[kCFreeTop], s);
      if (e1 != RS_OK || e2 != RS_OK || e3 != RS_OK) return RS_EHIP;
      reset_bound(t, std::max(cs[kCBaseKeys] + ts[kTTomb], cs[kCBaseLive]));
      return st;  // grow_for's message stays the last error
    }
    int64_t tombs = 0;
    RS_HIP(hipMemcpy(&tombs, t->d_scal + kTTomb, sizeof(int64_t), hipMemcpyDeviceToHost));
    // redo the reservation against the grown table (published under a new
    // tag: the scan's count may predate the growth)
    reset_bound(t, std::max(keys_need + tombs, rows_need));
    const int64_t tag2 = next_tag(t);
    RS_HIP(launch_rereserve(w, t->dev(), t->h_pin, tag2, s));
    t->bound_after[tag2 % rs_table::kTags] = t->live_bound;
  } else {
    t->live_bound = bound;
    t->bound_after[tag % rs_table::kTags] = t->live_bound;
  }
  RS_HIP(launch_compact_insert(values, n, t->dev(), w, occ_lists, t->ev(RS_K_COMPACT_INSERT),
                               t->ev(RS_K_INIT_ROWS), t->ev(RS_K_OCC), s));
  return RS_OK;
}

bool valid_dim(int d) { return d == 8 || d == 16 || d == 32 || d == 64 || d == 128 || d == 256; }

OptArgs make_opt(rs_table* t, const rs_opt_params* p) {
  OptArgs o{};
  o.opt = t->d.optimizer;
  o.lr = static_cast<float>(p->lr);
  o.eps = static_cast<float>(p->eps);
  o.beta1 = static_cast<float>(p->beta1);
  o.beta2 = static_cast<float>(p->beta2);
  o.omb1 = static_cast<float>(1.0 - p->beta1);
  o.omb2 = static_cast<float>(1.0 - p->beta2);
  o.bc1 = 1.0f;
  o.bc2 = 1.0f;
  o.wdlr = static_cast<float>(p->lr * p->weight_decay);
  o.lrt = static_cast<float>(p->lr);
  if (o.opt != RS_ADAGRAD && o.opt != RS_ADAGRAD_ROWWISE) {  // the Adam family
    t->adam_t += 1;
    const double bc1 = 1.0 - std::pow(p->beta1, static_cast<double>(t->adam_t));
    const double bc2 = 1.0 - std::pow(p->beta2, static_cast<double>(t->adam_t));
    o.bc1 = static_cast<float>(bc1);
    o.bc2 = static_cast<float>(bc2);
    o.lrt = static_cast<float>(p->lr * std::sqrt(bc2) / bc1);
  }
  return o;
}

rs_status check_ctx(const rs_table* t, const rs_ctx* c) {
  if (!t || !c) return fail(RS_EINVAL, "null table or context");
  if (c->table != t) return fail(RS_EINVAL, "context was filled by a forward on another table");
  if (c->priv[0] != 2) return fail(RS_EINVAL, "the context's forward has not been pooled");
  if (c->dim != t->d.dim) return fail(RS_EINVAL, "context dim mismatch");
  return RS_OK;
}

Work ctx_work(const rs_ctx* c) {
  Work w = make_work(c->workspace, make_layout(c->n, c->dim));
  w.offsets = c->offsets;
  return w;
}

// Rows of the upstream gradient of a forward (its output's rows).
int64_t grad_rows(const rs_ctx* c) { return padded_mode(c->mode) ? c->bags * c->pad_len : c->bags; }

}  // namespace

extern "C" {

int rs_version(void) { return RS_VERSION; }

const char* rs_last_error(void) { return g_last_error.c_str(); }

rs_status ht_create(const rs_table_desc* d, const rs_allocator* a, rs_stream stream, rs_table** out) {
  if (!d || !out) return fail(RS_EINVAL, "null descriptor or output");
  *out = nullptr;
  if (!valid_dim(d->dim)) return fail(RS_EINVAL, "dim must be 8, 16, 32, 64, 128 or 256");
  if (d->row_dtype != RS_F32 && d->row_dtype != RS_BF16) return fail(RS_EINVAL, "bad row_dtype");
  if (d->optimizer < RS_ADAGRAD || d->optimizer > RS_ADAM_ROWWISE) return fail(RS_EINVAL, "bad optimizer");
  if (!is_pow2(d->capacity_slots) || d->capacity_slots < 16 || d->capacity_slots > (int64_t(1) << 40))
    return fail(RS_EINVAL, "capacity_slots must be a power of two in [16, 2^40]");
  if (!(d->max_load > 0.0f && d->max_load <= 0.9f)) return fail(RS_EINVAL, "max_load must be in (0, 0.9]");
  if (!is_pow2(d->block_rows) || d->block_rows < 64) return fail(RS_EINVAL, "block_rows must be a power of two >= 64");
  if (!(d->init_lo <= d->init_hi) || !std::isfinite(d->init_lo) || !std::isfinite(d->init_hi))
    return fail(RS_EINVAL, "init range must be finite with lo <= hi");
  if (a && (!a->alloc || !a->free)) return fail(RS_EINVAL, "allocator needs both callbacks");
  hipStream_t s = static_cast<hipStream_t>(stream);
  rs_table* t = new (std::nothrow) rs_table;
  if (!t) return fail(RS_ENOMEM, "host allocation failed");
  t->d = *d;
  if (a) {
    t->a = *a;
    t->custom = true;
  }
  if (hipGetDevice(&t->device) != hipSuccess) {
    delete t;
    return fail(RS_EHIP, "hipGetDevice failed");
  }
  t->stride = static_cast<int64_t>(d->dim) * t->wbytes() + 4 * t->state_elems();
  if (d->evictable) {
    // {int64 key, uint32 clock of the last lookup} after the state
    t->meta_off = static_cast<int>((t->stride + 7) / 8 * 8);
    t->stride = t->meta_off + 12;
  }
  t->stride = (t->stride + 15) / 16 * 16;  // 16-byte row fragments
  t->cap = d->capacity_slots;
  t->limit = static_cast<int64_t>(std::floor(static_cast<double>(d->max_load) * static_cast<double>(t->cap)));
  t->slots = static_cast<Slot*>(t->alloc(sizeof(Slot) * static_cast<size_t>(t->cap)));
  t->d_scal = static_cast<int64_t*>(t->alloc(sizeof(int64_t) * kTScalars));
  if (!t->slots || !t->d_scal) {
    ht_destroy(t);
    return fail(RS_ENOMEM, "table allocation failed");
  }
  rs_status st = RS_OK;
  do {
    if (hipHostMalloc(reinterpret_cast<void**>(&t->h_pin), sizeof(int64_t) * 8, hipHostMallocDefault) != hipSuccess) {
      st = fail(RS_EHIP, "pinned read-back buffer allocation failed");
      break;
    }
    t->h_pin[0] = 0;
    for (int64_t& b : t->bound_after) b = -1;
    if (hipMemsetAsync(t->slots, 0, sizeof(Slot) * static_cast<size_t>(t->cap), s) != hipSuccess ||

        hipMemsetAsync(t->d_scal, 0, sizeof(int64_t) * kTScalars, s) != hipSuccess) {
      st = fail(RS_EHIP, "initial clear failed");
      break;
    }
    st = set_scalar(t, kTLimit, t->limit, s);
    if (st != RS_OK) break;
    if (t->custom) {
      // Blocks from the allocator: chunks of block_rows rows, at most as many
      // as the device's memory holds, addressed through a device table
      size_t total = 0;
      if (hipDeviceTotalMem(&total, t->device) != hipSuccess) {
        st = fail(RS_EHIP, "hipDeviceTotalMem failed");
        break;
      }
      t->chunk_bytes = static_cast<size_t>(d->block_rows) * static_cast<size_t>(t->stride);
      t->chunk_tab_cap = static_cast<int64_t>(total / t->chunk_bytes) + 1;
      t->d_chunk_tab = static_cast<uint8_t**>(t->alloc(sizeof(uint8_t*) * static_cast<size_t>(t->chunk_tab_cap)));
      if (!t->d_chunk_tab) {
        st = fail(RS_ENOMEM, "allocation of the Blocks chunk table failed");
        break;
      }
      if (hipStreamSynchronize(s) != hipSuccess) st = fail(RS_EHIP, "hipStreamSynchronize failed");
      break;
    }
    // reserve the Blocks address range: as many bytes as the device has
    hipMemAllocationProp prop = {};
    prop.type = hipMemAllocationTypePinned;
    prop.location.type = hipMemLocationTypeDevice;
    prop.location.id = t->device;
    size_t gran = 0, total = 0;
    if (hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityRecommended) != hipSuccess ||
        hipDeviceTotalMem(&total, t->device) != hipSuccess || gran == 0) {
      st = fail(RS_EHIP, "querying the virtual-memory granularity failed");
      break;
    }
    const size_t want = static_cast<size_t>(d->block_rows) * static_cast<size_t>(t->stride);
    t->chunk_bytes = (want + gran - 1) / gran * gran;
    t->va_size = (total + t->chunk_bytes - 1) / t->chunk_bytes * t->chunk_bytes;
    void* va = nullptr;
    if (hipMemAddressReserve(&va, t->va_size, 0, nullptr, 0) != hipSuccess) {
      (void)hipGetLastError();
      t->va_size = 0;
      st = fail(RS_ENOMEM, "reserving the Blocks address range failed");
      break;
    }
    t->va_base = static_cast<uint8_t*>(va);
    if (hipStreamSynchronize(s) != hipSuccess) st = fail(RS_EHIP, "hipStreamSynchronize failed");
  } while (false);
  if (st != RS_OK) {
    ht_destroy(t);
    return st;
  }
  *out = t;
  return RS_OK;
}

rs_status ht_destroy(rs_table* t) {
  if (!t) return RS_OK;
  rs_status st = RS_OK;
  if (hipDeviceSynchronize() != hipSuccess) st = fail(RS_EHIP, "hipDeviceSynchronize failed");
  if (st == RS_OK && t->d_scal) st = take_latched(t);
  t->release(t->slots);
  if (t->mapped) (void)hipMemUnmap(t->va_base, t->mapped);
  for (hipMemGenericAllocationHandle_t h : t->chunks) (void)hipMemRelease(h);
  if (t->va_base) (void)hipMemAddressFree(t->va_base, t->va_size);
  for (void* p : t->achunks) t->release(p);
  t->release(t->d_chunk_tab);
  t->release(t->d_scal);
  t->release(t->iws);
  t->release(t->free_rows);
  if (t->h_pin) (void)hipHostFree(t->h_pin);
  delete t;
  return st;
}

size_t lookup_workspace_bytes(int64_t n, int64_t /*bags*/, int64_t /*pad_len*/, const rs_table* t) {
  if (!t || n < 0) return 0;
  return make_layout(n, t->d.dim).total;
}

size_t ids_partition_workspace_bytes(int64_t n, int32_t nshards) {
  if (n < 0 || n > (int64_t(1) << 28) || nshards < 1 || nshards > kMaxShards) return 0;
  return make_part_layout(n, nshards).total;
}

rs_status ids_partition(const int64_t* values, int64_t n, int32_t nshards, uint64_t owner_seed, int64_t* keys_out,
                        int64_t* shard_offsets, int32_t* inverse, int64_t* info, void* workspace,
                        size_t workspace_bytes, rs_stream stream) {
  if (n < 0 || n > (int64_t(1) << 28)) return fail(RS_EINVAL, "n must be in [0, 2^28]");
  if (nshards < 1 || nshards > kMaxShards) return fail(RS_EINVAL, "nshards must be in [1, 1024]");
  if (!shard_offsets || !info) return fail(RS_EINVAL, "null shard_offsets or info");
  if (n > 0 && (!values || !keys_out || !inverse)) return fail(RS_EINVAL, "null values, keys_out or inverse");
  const PartLayout L = make_part_layout(n, nshards);
  if (!workspace || workspace_bytes < L.total) return fail(RS_EINVAL, "workspace missing or too small");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return fail(RS_EINVAL, "workspace must be 256-byte aligned");
  uint8_t* b = static_cast<uint8_t*>(workspace);
  const Work w = make_part_work(workspace, L, inverse);
  RS_HIP(launch_ids_partition(values, n, nshards, owner_seed, w, L.og, reinterpret_cast<int32_t*>(b + L.hist),
                              reinterpret_cast<int32_t*>(b + L.csum), reinterpret_cast<int32_t*>(b + L.kslot),
                              reinterpret_cast<int64_t*>(b + L.pscal), keys_out, shard_offsets, info,
                              static_cast<hipStream_t>(stream)));
  return RS_OK;
}

namespace {

// Host check of column offsets (and their boundary offsets / moduli): copies
// them back, so it synchronizes.
rs_status check_columns(const int64_t* col_off, int32_t ncols, int64_t n, const int64_t* bnd_off,
                        const int64_t* moduli, hipStream_t s) {
  std::vector<int64_t> co(static_cast<size_t>(ncols) + 1), aux(bnd_off ? ncols + 1 : moduli ? ncols : 0);
  RS_HIP(hipStreamSynchronize(s));
  RS_HIP(hipMemcpy(co.data(), col_off, sizeof(int64_t) * co.size(), hipMemcpyDeviceToHost));
  if (!aux.empty())
    RS_HIP(hipMemcpy(aux.data(), bnd_off ? bnd_off : moduli, sizeof(int64_t) * aux.size(), hipMemcpyDeviceToHost));
  if (co[0] != 0 || co[ncols] != n) return fail(RS_EINVAL, "column offsets must start at 0 and end at n");
  for (int32_t c = 0; c < ncols; ++c)
    if (co[c + 1] < co[c]) return fail(RS_EINVAL, "column offsets must be nondecreasing");
  if (bnd_off) {
    if (aux[0] != 0) return fail(RS_EINVAL, "boundary offsets must start at 0");
    for (int32_t c = 0; c < ncols; ++c)
      if (aux[c + 1] < aux[c]) return fail(RS_EINVAL, "boundary offsets must be nondecreasing");
  }
  if (moduli)
    for (int32_t c = 0; c < ncols; ++c)
      if (aux[c] <= 0) return fail(RS_EINVAL, "moduli must be > 0");
  return RS_OK;
}

}  // namespace

rs_status fused_bucketize(const float* values, int64_t n, const int64_t* col_offsets, int32_t ncols,
                          const float* boundaries, const int64_t* bnd_offsets, int64_t* out, int32_t validate,
                          rs_stream stream) {
  if (n < 0 || n >= (int64_t(1) << 40)) return fail(RS_EINVAL, "n must be in [0, 2^40)");
  if (ncols < 1 || !col_offsets || !bnd_offsets) return fail(RS_EINVAL, "need ncols >= 1 and both offset arrays");
  if (n > 0 && (!values || !out)) return fail(RS_EINVAL, "null values or out");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (validate) {
    const rs_status st = check_columns(col_offsets, ncols, n, bnd_offsets, nullptr, s);
    if (st != RS_OK) return st;
  }
  RS_HIP(launch_bucketize(values, n, col_offsets, ncols, boundaries, bnd_offsets, out, s));
  return RS_OK;
}

rs_status fused_mod(const int64_t* values, int64_t n, const int64_t* col_offsets, int32_t ncols,
                    const int64_t* moduli, int64_t* out, int32_t validate, rs_stream stream) {
  if (n < 0 || n >= (int64_t(1) << 40)) return fail(RS_EINVAL, "n must be in [0, 2^40)");
  if (ncols < 1 || !col_offsets || !moduli) return fail(RS_EINVAL, "need ncols >= 1, offsets and moduli");
  if (n > 0 && (!values || !out)) return fail(RS_EINVAL, "null values or out");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (validate) {
    const rs_status st = check_columns(col_offsets, ncols, n, nullptr, moduli, s);
    if (st != RS_OK) return st;
  }
  RS_HIP(launch_mod(values, n, col_offsets, ncols, moduli, out, s));
  return RS_OK;
}

rs_status ht_find_or_insert(rs_table* t, const int64_t* keys, int64_t n, int64_t* rows_out, int64_t* n_inserted_dev,
                            rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (n < 0 || n > (int64_t(1) << 28)) return fail(RS_EINVAL, "n must be in [0, 2^28]");
  if (n > 0 && (!keys || !rows_out)) return fail(RS_EINVAL, "null keys or rows_out");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n == 0) {
    if (n_inserted_dev) RS_HIP(hipMemsetAsync(n_inserted_dev, 0, sizeof(int64_t), s));
    return RS_OK;
  }
  const Layout L = make_layout(n, t->d.dim);
  if (t->iws_bytes < L.total) {
    RS_HIP(hipStreamSynchronize(s));
    t->release(t->iws);
    t->iws = t->alloc(L.total);
    t->iws_bytes = t->iws ? L.total : 0;
    if (!t->iws) return fail(RS_ENOMEM, "allocation of the insert workspace failed");
  }
  const Work w = make_work(t->iws, L);
  t->clock += 1;  // one lookup call
  rs_status st = dedup_and_insert(t, keys, n, w, false, s);
  if (st != RS_OK) return st;
  RS_HIP(launch_map_rows(w, n, rows_out, n_inserted_dev, s));
  return RS_OK;
}

rs_status ht_find(rs_table* t, const int64_t* keys, int64_t n, int64_t* rows_out, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (n < 0) return fail(RS_EINVAL, "n < 0");
  if (n > 0 && (!keys || !rows_out)) return fail(RS_EINVAL, "null keys or rows_out");
  RS_HIP(launch_find(t->dev(), keys, n, rows_out, static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status ht_size(rs_table* t, int64_t* live_host, rs_stream stream) {
  if (!t || !live_host) return fail(RS_EINVAL, "null table or output");
  hipStream_t s = static_cast<hipStream_t>(stream);
  RS_HIP(hipStreamSynchronize(s));
  int64_t ts[kTScalars];
  RS_HIP(hipMemcpy(ts, t->d_scal, sizeof(ts), hipMemcpyDeviceToHost));
  *live_host = ts[kTKeys];
  reset_bound(t, std::max(ts[kTKeys] + ts[kTTomb], ts[kTLive]));
  return take_latched(t);
}

rs_status ht_evict(rs_table* t, uint32_t max_age, int64_t* n_evicted_host, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (t->meta_off < 0) return fail(RS_EINVAL, "the table was created without eviction (evictable = 0)");
  if (t->rows_prov >= (int64_t(1) << 31)) return fail(RS_EINVAL, "eviction counts rows in 32 bits: fewer than 2^31 rows");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t nb = std::max<int64_t>(1, (t->rows_prov + kEvictRows - 1) / kEvictRows);
  int32_t* bcount = static_cast<int32_t*>(t->alloc(sizeof(int32_t) * static_cast<size_t>(nb + 1)));
  if (!bcount) return fail(RS_ENOMEM, "allocation of the eviction counts failed");
  rs_status st = RS_OK;
  if (t->rows_prov > 0) {
    const hipError_t e = launch_evict(t->dev(), t->rows_prov, max_age, bcount, s);
    if (e != hipSuccess) st = fail(RS_EHIP, std::string("eviction launch: ") + hipGetErrorString(e));
  }
  int64_t ts[kTScalars] = {};
  int32_t n = 0;
  if (st == RS_OK && (hipStreamSynchronize(s) != hipSuccess ||
                      (t->rows_prov > 0 && hipMemcpy(&n, bcount + nb, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess) ||
                      hipMemcpy(ts, t->d_scal, sizeof(ts), hipMemcpyDeviceToHost) != hipSuccess))
    st = fail(RS_EHIP, "eviction read-back failed");
  t->release(bcount);
  if (st != RS_OK) return st;
  reset_bound(t, std::max(ts[kTKeys] + ts[kTTomb], ts[kTLive]));
  if (n_evicted_host) *n_evicted_host = n;
  return take_latched(t);
}

rs_status ht_compact(rs_table* t, int64_t* moved_host, int64_t* bytes_released_host, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (t->meta_off < 0) return fail(RS_EINVAL, "the table was created without eviction (evictable = 0)");
  hipStream_t s = static_cast<hipStream_t>(stream);
  RS_HIP(hipStreamSynchronize(s));
  int64_t ts[kTScalars];
  RS_HIP(hipMemcpy(ts, t->d_scal, sizeof(ts), hipMemcpyDeviceToHost));
  const int64_t L = ts[kTKeys], hw = ts[kTLive];
  int64_t moved = 0;
  if (hw > L) {
    const int64_t nb = (hw + kEvictRows - 1) / kEvictRows;
    int32_t* cnt = static_cast<int32_t*>(t->alloc(sizeof(int32_t) * 2 * static_cast<size_t>(nb + 1)));
    int64_t* lists = static_cast<int64_t*>(t->alloc(sizeof(int64_t) * 2 * static_cast<size_t>(hw - L)));
    rs_status st = RS_OK;
    if (!cnt || !lists) {
      st = fail(RS_ENOMEM, "allocation of the compaction lists failed");
    } else {
      const hipError_t e = launch_compact_rows(t->dev(), L, hw, cnt, cnt + nb + 1, lists, lists + (hw - L), s);
      int32_t h[2] = {0, 0};
      if (e != hipSuccess || hipStreamSynchronize(s) != hipSuccess ||
          hipMemcpy(&h[0], cnt + nb, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess ||
          hipMemcpy(&h[1], cnt + nb + 1 + nb, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess)
        st = fail(RS_EHIP, "compaction failed");
      moved = std::min(h[0], h[1]);
    }
    t->release(cnt);
    t->release(lists);
    if (st != RS_OK) return st;
  }
  // give back the Blocks memory past row L (whole chunks)
  int64_t released = 0;
  if (t->custom) {
    const size_t keep = static_cast<size_t>((L + t->d.block_rows - 1) / t->d.block_rows);
    while (t->achunks.size() > keep) {
      t->release(t->achunks.back());
      t->achunks.pop_back();
      released += static_cast<int64_t>(t->chunk_bytes);
    }
    t->rows_prov = static_cast<int64_t>(t->achunks.size()) * t->d.block_rows;
  } else {
    const size_t need = static_cast<size_t>(L) * static_cast<size_t>(t->stride);
    const size_t keep = (need + t->chunk_bytes - 1) / t->chunk_bytes;
    while (t->chunks.size() > keep) {
      const size_t off = (t->chunks.size() - 1) * t->chunk_bytes;
      if (hipMemUnmap(t->va_base + off, t->chunk_bytes) != hipSuccess ||
          hipMemRelease(t->chunks.back()) != hipSuccess) {
        (void)hipGetLastError();
        return fail(RS_EHIP, "unmapping a Blocks chunk failed");
      }
      t->chunks.pop_back();
      t->mapped -= t->chunk_bytes;
      released += static_cast<int64_t>(t->chunk_bytes);
    }
    t->rows_prov = static_cast<int64_t>(t->mapped / static_cast<size_t>(t->stride));
  }
  rs_status st = set_scalar(t, kTRowCap, t->rows_prov, s);
  if (st != RS_OK) return st;
  RS_HIP(hipStreamSynchronize(s));
  reset_bound(t, std::max(L + ts[kTTomb], L));
  if (moved_host) *moved_host = moved;
  if (bytes_released_host) *bytes_released_host = released;
  return take_latched(t);
}

rs_status rs_table_check(rs_table* t, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  RS_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  return take_latched(t);
}

rs_status ht_capacity(const rs_table* t, int64_t* slots_host) {
  if (!t || !slots_host) return fail(RS_EINVAL, "null table or output");
  *slots_host = t->cap;
  return RS_OK;
}

rs_status ht_export(rs_table* t, int64_t* keys, int64_t* rows, int64_t cap, int64_t* n_dev, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (cap < 0 || (cap > 0 && (!keys || !rows))) return fail(RS_EINVAL, "bad output arrays");
  RS_HIP(launch_export(t->dev(), t->cap, keys, rows, cap, n_dev, static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status ht_read_rows(rs_table* t, const int64_t* rows, int64_t n, float* w_out, float* state_out, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (n < 0 || (n > 0 && !rows)) return fail(RS_EINVAL, "bad rows");
  if (t->rows_prov == 0) {
    // no Blocks yet: every row is out of range
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (n > 0 && w_out) RS_HIP(hipMemsetAsync(w_out, 0xFF, sizeof(float) * n * t->d.dim, s));
    if (n > 0 && state_out) RS_HIP(hipMemsetAsync(state_out, 0xFF, sizeof(float) * n * t->state_elems(), s));
    return RS_OK;
  }
  RS_HIP(launch_read_rows(t->dev(), rows, n, w_out, state_out, static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status ht_reserve(rs_table* t, int64_t live_upper_bound, rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (live_upper_bound < 0) return fail(RS_EINVAL, "negative bound");
  hipStream_t s = static_cast<hipStream_t>(stream);
  RS_HIP(hipStreamSynchronize(s));
  int64_t c = t->cap;
  while (static_cast<double>(live_upper_bound) > static_cast<double>(t->d.max_load) * static_cast<double>(c)) c <<= 1;
  if (c != t->cap) {
    rs_status st = rehash(t, c, s);
    if (st != RS_OK) return st;
  }
  rs_status st = provision_rows(t, live_upper_bound, s);
  if (st != RS_OK) return st;
  RS_HIP(hipStreamSynchronize(s));
  return take_latched(t);
}

rs_status lookup_prepare(rs_table* t, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags,
                         int32_t mode, int64_t pad_len, rs_ctx* ctx, int32_t validate, rs_stream stream) {
  if (!t || !ctx) return fail(RS_EINVAL, "null table or context");
  if (n < 0 || n > (int64_t(1) << 28)) return fail(RS_EINVAL, "n must be in [0, 2^28]");
  if (bags < 0 || bags >= (int64_t(1) << 31)) return fail(RS_EINVAL, "bags must be in [0, 2^31)");
  if (mode != RS_POOL_SUM && mode != RS_POOL_MEAN && !padded_mode(mode)) return fail(RS_EINVAL, "bad pooling mode");
  if (padded_mode(mode)) {
    if (pad_len <= 0) return fail(RS_EINVAL, "pad_len must be > 0 for the padded modes");
    if (bags * pad_len >= (int64_t(1) << 31)) return fail(RS_EINVAL, "bags * pad_len must be < 2^31");
  }
  if (!offsets || (n > 0 && !values)) return fail(RS_EINVAL, "null input");
  const Layout L = make_layout(n, t->d.dim);
  if (!ctx->workspace || ctx->workspace_bytes < L.total) return fail(RS_EINVAL, "workspace missing or too small");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (validate) {
    std::vector<int64_t> h(static_cast<size_t>(bags + 1));
    RS_HIP(hipStreamSynchronize(s));
    RS_HIP(hipMemcpy(h.data(), offsets, sizeof(int64_t) * (bags + 1), hipMemcpyDeviceToHost));
    if (h[0] != 0 || h[bags] != n) return fail(RS_EINVAL, "offsets must start at 0 and end at n");
    for (int64_t g = 0; g < bags; ++g)
      if (h[g + 1] < h[g]) return fail(RS_EINVAL, "offsets must be nondecreasing");
  }
  const Work w = make_work(ctx->workspace, L);
  ctx->table = nullptr;  // published only once the work has been enqueued
  ctx->priv[0] = 0;      // 1: prepared, 2: pooled
  ctx->unique = w.unique;
  ctx->inverse = w.inverse;
  ctx->rows = w.rows;
  ctx->scalars = w.scal;
  ctx->offsets = offsets;
  ctx->n = n;
  ctx->bags = bags;
  ctx->pad_len = padded_mode(mode) ? pad_len : 0;
  ctx->mode = mode;
  ctx->dim = t->d.dim;
  t->clock += 1;  // one lookup call
  rs_status st = dedup_and_insert(t, values, n, w, true, s);
  if (st != RS_OK) return st;
  ctx->priv[0] = 1;
  ctx->table = t;
  return RS_OK;
}

rs_status lookup_pool_prepared(rs_table* t, rs_ctx* ctx, void* out, uint8_t* mask, rs_stream stream) {
  if (!t || !ctx) return fail(RS_EINVAL, "null table or context");
  if (ctx->table != t || ctx->priv[0] < 1) return fail(RS_EINVAL, "context was not prepared on this table");
  if (ctx->bags > 0 && !out) return fail(RS_EINVAL, "null output");
  if (padded_mode(ctx->mode) && ctx->bags > 0 && !mask) return fail(RS_EINVAL, "null mask");
  const Work w = ctx_work(ctx);
  RS_HIP(launch_pool(t->dev(), w, ctx->offsets, ctx->n, ctx->bags, ctx->mode, ctx->pad_len, out, mask,
                     t->ev(RS_K_POOL), static_cast<hipStream_t>(stream)));
  ctx->priv[0] = 2;
  return RS_OK;
}

rs_status lookup_pool_fwd(rs_table* t, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags,
                          int32_t mode, int64_t pad_len, void* out, uint8_t* mask, rs_ctx* ctx, int32_t validate,
                          rs_stream stream) {
  if (bags > 0 && !out) return fail(RS_EINVAL, "null output");
  if (padded_mode(mode) && bags > 0 && !mask) return fail(RS_EINVAL, "null mask");
  rs_status st = lookup_prepare(t, values, offsets, n, bags, mode, pad_len, ctx, validate, stream);
  if (st != RS_OK) return st;
  return lookup_pool_prepared(t, ctx, out, mask, stream);
}

rs_status lookup_pool_bwd(rs_table* t, const rs_ctx* ctx, const void* grad_out, float* grad_unique, rs_stream stream) {
  rs_status st = check_ctx(t, ctx);
  if (st != RS_OK) return st;
  if (ctx->n > 0 && (!grad_out || !grad_unique)) return fail(RS_EINVAL, "null gradient");
  const Work w = ctx_work(ctx);
  RS_HIP(launch_bwd(t->dev(), w, grad_rows(ctx), ctx->n, ctx->mode, grad_out, grad_unique, nullptr,
                    t->ev(RS_K_OCC_LIST), t->ev(RS_K_BWD_SHORT), t->ev(RS_K_BWD_LONG), static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status sparse_opt_step(rs_table* t, const rs_ctx* ctx, const float* grad_unique, const rs_opt_params* p,
                          rs_stream stream) {
  rs_status st = check_ctx(t, ctx);
  if (st != RS_OK) return st;
  if (!p) return fail(RS_EINVAL, "null optimizer parameters");
  if (ctx->n > 0 && !grad_unique) return fail(RS_EINVAL, "null grad_unique");
  const OptArgs o = make_opt(t, p);
  const Work w = ctx_work(ctx);
  RS_HIP(launch_opt(t->dev(), w, ctx->n, grad_unique, o, t->ev(RS_K_OPT), static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status lookup_pool_bwd_opt(rs_table* t, const rs_ctx* ctx, const void* grad_out, const rs_opt_params* p,
                              rs_stream stream) {
  rs_status st = check_ctx(t, ctx);
  if (st != RS_OK) return st;
  if (!p) return fail(RS_EINVAL, "null optimizer parameters");
  if (ctx->n > 0 && !grad_out) return fail(RS_EINVAL, "null gradient");
  const OptArgs o = make_opt(t, p);
  const Work w = ctx_work(ctx);
  RS_HIP(launch_bwd(t->dev(), w, grad_rows(ctx), ctx->n, ctx->mode, grad_out, nullptr, &o, t->ev(RS_K_OCC_LIST), t->ev(RS_K_BWD_SHORT),
                    t->ev(RS_K_BWD_LONG), static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status rs_bandwidth_probe(int32_t kind, void* a, int64_t a_bytes, void* b, int64_t b_bytes, const int64_t* idx,
                             int64_t n, int32_t row_bytes, rs_stream stream) {
  if (!a || a_bytes <= 0 || n < 0) return fail(RS_EINVAL, "null or empty buffer a, or n < 0");
  const bool rows = kind == RS_PROBE_GATHER || kind == RS_PROBE_RMW;
  if (kind < RS_PROBE_READ || kind > RS_PROBE_RMW) return fail(RS_EINVAL, "bad probe kind");
  if (!rows) {
    if (n % 16 != 0 || n > a_bytes) return fail(RS_EINVAL, "n must be a multiple of 16 and at most a_bytes");
    if ((kind == RS_PROBE_READ && (!b || b_bytes < 4)) || (kind == RS_PROBE_COPY && (!b || n > b_bytes)))
      return fail(RS_EINVAL, "buffer b missing or too small");
  } else {
    if (row_bytes <= 0 || row_bytes % 16 != 0 || probe_lanes(row_bytes / 16) == 0 || row_bytes > a_bytes)
      return fail(RS_EINVAL, "row_bytes must be 16 * 2^k * c (c <= 4, 2^k <= 64) and at most a_bytes");
    if (!idx) return fail(RS_EINVAL, "null idx");
    if (kind == RS_PROBE_GATHER && (!b || n > b_bytes / row_bytes)) return fail(RS_EINVAL, "buffer b too small");
  }
  if (n == 0) return RS_OK;
  RS_HIP(launch_probe(kind, a, a_bytes, b, idx, n, row_bytes, static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status rs_set_kernel_events(rs_table* t, int32_t kernel, void* start_event, void* stop_event) {
  if (!t || kernel < 0 || kernel >= RS_K_COUNT) return fail(RS_EINVAL, "bad table or kernel id");
  t->kev[kernel][0] = static_cast<hipEvent_t>(start_event);
  t->kev[kernel][1] = static_cast<hipEvent_t>(stop_event);
  return RS_OK;
}

}  // extern "C"

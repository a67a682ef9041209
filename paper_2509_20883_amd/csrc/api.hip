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

int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

// Workspace layout of one forward: every array sized by the upper bound n.
struct Layout {
  size_t slot_of, occ_rank, inverse, unique, uslot, ucount, seg, rows, isnew, occ_ref, chunk_u, bsum, scal,
      gpart, total;
};

Layout make_layout(int64_t n, int dim) {
  const size_t n1 = static_cast<size_t>(n > 0 ? n : 1);
  const size_t nch = n1 / kChunk + 2;
  const size_t nb = n1 / kScanTile + 2;
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.slot_of = take(4 * n1);
  L.occ_rank = take(4 * n1);
  L.inverse = take(4 * n1);
  L.unique = take(8 * n1);
  L.uslot = take(4 * n1);
  L.ucount = take(4 * n1);
  L.seg = take(4 * (n1 + 1));
  L.rows = take(8 * n1);
  L.isnew = take(4 * n1);
  L.occ_ref = take(4 * n1);
  L.chunk_u = take(4 * nch);
  L.bsum = take(4 * nb);
  L.scal = take(8 * kCScalars);
  L.gpart = take(4 * nch * static_cast<size_t>(dim));
  L.total = off;
  return L;
}

Work make_work(void* base, const Layout& L) {
  uint8_t* b = static_cast<uint8_t*>(base);
  Work w;
  w.slot_of = reinterpret_cast<int32_t*>(b + L.slot_of);
  w.occ_rank = reinterpret_cast<int32_t*>(b + L.occ_rank);
  w.inverse = reinterpret_cast<int32_t*>(b + L.inverse);
  w.unique = reinterpret_cast<int64_t*>(b + L.unique);
  w.uslot = reinterpret_cast<int32_t*>(b + L.uslot);
  w.ucount = reinterpret_cast<int32_t*>(b + L.ucount);
  w.seg = reinterpret_cast<int32_t*>(b + L.seg);
  w.rows = reinterpret_cast<int64_t*>(b + L.rows);
  w.isnew = reinterpret_cast<int32_t*>(b + L.isnew);
  w.occ_ref = reinterpret_cast<int32_t*>(b + L.occ_ref);
  w.chunk_u = reinterpret_cast<int32_t*>(b + L.chunk_u);
  w.bsum = reinterpret_cast<int32_t*>(b + L.bsum);
  w.scal = reinterpret_cast<int64_t*>(b + L.scal);
  w.gpart = reinterpret_cast<float*>(b + L.gpart);
  return w;
}

const char* err_text(int bits) {
  if (bits & kErrKey) return "a reserved key (INT64_MIN or INT64_MIN+1) was in the input";
  if (bits & kErrFull) return "the table is full (auto_grow is off): some keys were not inserted";
  if (bits & kErrScratch) return "dedup scratch table overflow";
  if (bits & kErrProbe) return "IDMap probe found no free slot";
  return "device error";
}

rs_status err_status(int bits) {
  if (bits & kErrKey) return RS_EKEY;
  if (bits & kErrFull) return RS_EFULL;
  return RS_EHIP;
}

}  // namespace

struct rs_table {
  rs_table_desc d{};
  rs_allocator a{};
  bool custom = false;
  int device = 0;
  // IDMap
  Slot* slots = nullptr;
  int64_t cap = 0;
  int64_t limit = 0;  // floor(max_load * cap)
  // Blocks
  std::vector<uint8_t*> blocks;
  uint8_t** d_blocks = nullptr;
  int64_t stride = 0;
  int block_shift = 0;
  int64_t rows_prov = 0;
  // device scalars
  int64_t* d_scal = nullptr;
  // dedup scratch
  unsigned long long* s_key = nullptr;
  unsigned int* s_first = nullptr;
  unsigned int* s_cnt = nullptr;
  int32_t* s_uid = nullptr;
  int64_t s_cap = 0;
  // host view of the live count: an upper bound, refreshed from an
  // asynchronous read-back when one has completed
  int64_t live_bound = 0;
  int64_t* h_pin = nullptr;
  hipEvent_t rb_ev = nullptr;
  bool rb_pending = false;
  int64_t rb_bound = 0;
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
  int nstate() const { return d.optimizer == RS_ADAM ? 2 : 1; }
  int wbytes() const { return d.row_dtype == RS_BF16 ? 2 : 4; }

  TableDev dev() const {
    TableDev t;
    t.slots = slots;
    t.cap_mask = static_cast<uint64_t>(cap - 1);
    t.store.blocks = d_blocks;
    t.store.shift = block_shift;
    t.store.mask = d.block_rows - 1;
    t.store.stride = stride;
    t.scal = d_scal;
    t.dim = d.dim;
    t.row_dtype = d.row_dtype;
    t.nstate = nstate();
    t.seed = d.seed;
    t.lo = d.init_lo;
    t.span = d.init_hi - d.init_lo;  // fp32 subtraction
    return t;
  }
  Scratch scratch() const { return Scratch{s_key, s_first, s_cnt, s_uid, static_cast<uint64_t>(s_cap - 1)}; }
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

// Ensure the dedup scratch has >= 2n slots (load <= 0.5); it is cleared once
// here and then returned to empty by every call that used it.
rs_status ensure_scratch(rs_table* t, int64_t n, hipStream_t s) {
  int64_t want = 4096;
  while (want < 2 * n) want <<= 1;
  if (t->s_cap >= want) return RS_OK;
  RS_HIP(hipStreamSynchronize(s));
  t->release(t->s_key);
  t->release(t->s_first);
  t->release(t->s_cnt);
  t->release(t->s_uid);
  t->s_key = static_cast<unsigned long long*>(t->alloc(8 * want));
  t->s_first = static_cast<unsigned int*>(t->alloc(4 * want));
  t->s_cnt = static_cast<unsigned int*>(t->alloc(4 * want));
  t->s_uid = static_cast<int32_t*>(t->alloc(4 * want));
  if (!t->s_key || !t->s_first || !t->s_cnt || !t->s_uid) {
    t->s_cap = 0;
    return fail(RS_ENOMEM, "allocation of the dedup scratch failed");
  }
  t->s_cap = want;
  RS_HIP(hipMemsetAsync(t->s_key, 0, 8 * want, s));
  RS_HIP(hipMemsetAsync(t->s_first, 0xFF, 4 * want, s));
  RS_HIP(hipMemsetAsync(t->s_cnt, 0, 4 * want, s));
  return RS_OK;
}

// Add Blocks chunks until `rows` rows fit.
rs_status provision_rows(rs_table* t, int64_t rows, hipStream_t s) {
  if (rows <= t->rows_prov) return RS_OK;
  const int64_t br = t->d.block_rows;
  const int64_t need_blocks = (rows + br - 1) / br;
  if (need_blocks > kMaxBlocks) return fail(RS_ENOMEM, "too many Blocks chunks (raise block_rows)");
  const size_t first_new = t->blocks.size();
  while (static_cast<int64_t>(t->blocks.size()) < need_blocks) {
    void* p = t->alloc(static_cast<size_t>(br) * static_cast<size_t>(t->stride));
    if (!p) return fail(RS_ENOMEM, "allocation of a Blocks chunk failed");
    t->blocks.push_back(static_cast<uint8_t*>(p));
  }
  // entries past the old count are read by no kernel yet: a plain copy is safe
  RS_HIP(hipMemcpy(t->d_blocks + first_new, t->blocks.data() + first_new,
                   sizeof(uint8_t*) * (t->blocks.size() - first_new), hipMemcpyHostToDevice));
  t->rows_prov = static_cast<int64_t>(t->blocks.size()) * br;
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
  RS_HIP(hipStreamSynchronize(s));
  t->release(old);
  return RS_OK;
}

// Grow (when allowed) so that `live_need` keys fit the IDMap and the Blocks.
rs_status grow_for(rs_table* t, int64_t live_need, hipStream_t s) {
  if (t->d.auto_grow) {
    int64_t c = t->cap;
    while (static_cast<double>(live_need) > static_cast<double>(t->d.max_load) * static_cast<double>(c)) c <<= 1;
    if (c != t->cap) {
      rs_status st = rehash(t, c, s);
      if (st != RS_OK) return st;
    }
    const int64_t headroom = live_need + live_need / 8 + t->d.block_rows;
    return provision_rows(t, headroom, s);
  }
  return provision_rows(t, std::min(live_need, t->limit), s);
}

void refresh_bound(rs_table* t) {
  if (t->rb_pending && hipEventQuery(t->rb_ev) == hipSuccess) {
    t->rb_pending = false;
    const int64_t exact = *t->h_pin;
    t->live_bound = exact + (t->live_bound - t->rb_bound);
  }
}

void start_readback(rs_table* t, hipStream_t s) {
  if (t->rb_pending) return;
  if (hipMemcpyAsync(t->h_pin, t->d_scal + kTLive, sizeof(int64_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipEventRecord(t->rb_ev, s) != hipSuccess) {
    (void)hipGetLastError();
    return;
  }
  t->rb_pending = true;
  t->rb_bound = t->live_bound;
}

// Dedup `values` into w, then find-or-insert the unique keys (growing the
// table first when it may not have room).
rs_status dedup_and_insert(rs_table* t, const int64_t* values, int64_t n, const Work& w, hipStream_t s) {
  rs_status st = ensure_scratch(t, n, s);
  if (st != RS_OK) return st;
  const Scratch sc = t->scratch();
  RS_HIP(launch_dedup(values, n, sc, w, reinterpret_cast<int*>(t->d_scal + kTErr), t->ev(RS_K_DEDUP_LOCAL),
                      t->ev(RS_K_DEDUP_COMPACT), s));
  RS_HIP(launch_seg_scan(w, n, sc, t->d.dim, s));
  refresh_bound(t);
  const int64_t bound = t->live_bound + n;
  if (bound > t->limit || bound > t->rows_prov) {
    // exact decision: read back U and live (one synchronization)
    RS_HIP(hipStreamSynchronize(s));
    int64_t U = 0, live = 0;
    RS_HIP(hipMemcpy(&U, w.scal + kCU, sizeof(int64_t), hipMemcpyDeviceToHost));
    RS_HIP(hipMemcpy(&live, t->d_scal + kTLive, sizeof(int64_t), hipMemcpyDeviceToHost));
    t->rb_pending = false;
    t->live_bound = live;
    st = grow_for(t, live + U, s);
    if (st != RS_OK) return st;
    t->live_bound = live + U;
  } else {
    t->live_bound = bound;
  }
  const TableDev td = t->dev();
  RS_HIP(launch_idmap_probe(td, w, n, t->ev(RS_K_IDMAP_PROBE), s));
  RS_HIP(launch_idmap_insert(td, w, n, t->ev(RS_K_IDMAP_INSERT), s));
  start_readback(t, s);
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
  if (o.opt == RS_ADAM) {
    t->adam_t += 1;
    o.bc1 = static_cast<float>(1.0 - std::pow(p->beta1, static_cast<double>(t->adam_t)));
    o.bc2 = static_cast<float>(1.0 - std::pow(p->beta2, static_cast<double>(t->adam_t)));
  }
  return o;
}

rs_status check_ctx(const rs_table* t, const rs_ctx* c) {
  if (!t || !c) return fail(RS_EINVAL, "null table or context");
  if (c->table != t) return fail(RS_EINVAL, "context was filled by a forward on another table");
  if (c->dim != t->d.dim) return fail(RS_EINVAL, "context dim mismatch");
  return RS_OK;
}

Work ctx_work(const rs_ctx* c) { return make_work(c->workspace, make_layout(c->n, c->dim)); }

}  // namespace

extern "C" {

int rs_version(void) { return RS_VERSION; }

const char* rs_last_error(void) { return g_last_error.c_str(); }

rs_status ht_create(const rs_table_desc* d, const rs_allocator* a, rs_stream stream, rs_table** out) {
  if (!d || !out) return fail(RS_EINVAL, "null descriptor or output");
  *out = nullptr;
  if (!valid_dim(d->dim)) return fail(RS_EINVAL, "dim must be 8, 16, 32, 64, 128 or 256");
  if (d->row_dtype != RS_F32 && d->row_dtype != RS_BF16) return fail(RS_EINVAL, "bad row_dtype");
  if (d->optimizer != RS_ADAGRAD && d->optimizer != RS_ADAM) return fail(RS_EINVAL, "bad optimizer");
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
  t->stride = static_cast<int64_t>(d->dim) * (t->wbytes() + 4 * t->nstate());
  t->block_shift = ilog2(d->block_rows);
  t->cap = d->capacity_slots;
  t->limit = static_cast<int64_t>(std::floor(static_cast<double>(d->max_load) * static_cast<double>(t->cap)));
  t->slots = static_cast<Slot*>(t->alloc(sizeof(Slot) * static_cast<size_t>(t->cap)));
  t->d_blocks = static_cast<uint8_t**>(t->alloc(sizeof(uint8_t*) * kMaxBlocks));
  t->d_scal = static_cast<int64_t*>(t->alloc(sizeof(int64_t) * kTScalars));
  if (!t->slots || !t->d_blocks || !t->d_scal) {
    ht_destroy(t);
    return fail(RS_ENOMEM, "table allocation failed");
  }
  rs_status st = RS_OK;
  do {
    if (hipHostMalloc(reinterpret_cast<void**>(&t->h_pin), sizeof(int64_t) * 8, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&t->rb_ev, hipEventDisableTiming) != hipSuccess) {
      st = fail(RS_EHIP, "pinned read-back buffer or event creation failed");
      break;
    }
    if (hipMemsetAsync(t->slots, 0, sizeof(Slot) * static_cast<size_t>(t->cap), s) != hipSuccess ||
        hipMemsetAsync(t->d_blocks, 0, sizeof(uint8_t*) * kMaxBlocks, s) != hipSuccess ||
        hipMemsetAsync(t->d_scal, 0, sizeof(int64_t) * kTScalars, s) != hipSuccess) {
      st = fail(RS_EHIP, "initial clear failed");
      break;
    }
    st = set_scalar(t, kTLimit, t->limit, s);
    if (st != RS_OK) break;
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
  for (uint8_t* b : t->blocks) t->release(b);
  t->release(t->d_blocks);
  t->release(t->d_scal);
  t->release(t->s_key);
  t->release(t->s_first);
  t->release(t->s_cnt);
  t->release(t->s_uid);
  t->release(t->iws);
  if (t->h_pin) (void)hipHostFree(t->h_pin);
  if (t->rb_ev) (void)hipEventDestroy(t->rb_ev);
  delete t;
  return st;
}

size_t lookup_workspace_bytes(int64_t n, int64_t /*bags*/, int64_t /*pad_len*/, const rs_table* t) {
  if (!t || n < 0) return 0;
  return make_layout(n, t->d.dim).total;
}

rs_status ht_find_or_insert(rs_table* t, const int64_t* keys, int64_t n, int64_t* rows_out, int64_t* n_inserted_dev,
                            rs_stream stream) {
  if (!t) return fail(RS_EINVAL, "null table");
  if (n < 0 || n > (int64_t(1) << 30)) return fail(RS_EINVAL, "n must be in [0, 2^30]");
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
  rs_status st = dedup_and_insert(t, keys, n, w, s);
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
  RS_HIP(hipMemcpy(live_host, t->d_scal + kTLive, sizeof(int64_t), hipMemcpyDeviceToHost));
  t->rb_pending = false;
  t->live_bound = *live_host;
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
    if (n > 0 && state_out) RS_HIP(hipMemsetAsync(state_out, 0xFF, sizeof(float) * n * t->d.dim * t->nstate(), s));
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

rs_status lookup_pool_fwd(rs_table* t, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags,
                          int32_t mode, int64_t pad_len, void* out, uint8_t* mask, rs_ctx* ctx, int32_t validate,
                          rs_stream stream) {
  if (!t || !ctx) return fail(RS_EINVAL, "null table or context");
  if (n < 0 || n > (int64_t(1) << 30)) return fail(RS_EINVAL, "n must be in [0, 2^30]");
  if (bags < 0 || bags >= (int64_t(1) << 31)) return fail(RS_EINVAL, "bags must be in [0, 2^31)");
  if (mode != RS_POOL_SUM && mode != RS_POOL_MEAN && mode != RS_POOL_NONE) return fail(RS_EINVAL, "bad pooling mode");
  if (mode == RS_POOL_NONE) {
    if (pad_len <= 0) return fail(RS_EINVAL, "pad_len must be > 0 for RS_POOL_NONE");
    if (bags * pad_len >= (int64_t(1) << 31)) return fail(RS_EINVAL, "bags * pad_len must be < 2^31");
    if (bags > 0 && !mask) return fail(RS_EINVAL, "null mask");
  }
  if (!offsets || (n > 0 && !values) || (bags > 0 && !out)) return fail(RS_EINVAL, "null input or output");
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
  ctx->table = nullptr;  // published only once the forward has been enqueued
  ctx->unique = w.unique;
  ctx->inverse = w.inverse;
  ctx->rows = w.rows;
  ctx->scalars = w.scal;
  ctx->offsets = offsets;
  ctx->n = n;
  ctx->bags = bags;
  ctx->pad_len = mode == RS_POOL_NONE ? pad_len : 0;
  ctx->mode = mode;
  ctx->dim = t->d.dim;
  rs_status st = dedup_and_insert(t, values, n, w, s);
  if (st != RS_OK) return st;
  RS_HIP(launch_pool(t->dev(), w, offsets, n, bags, mode, ctx->pad_len, out, mask, t->ev(RS_K_POOL), s));
  ctx->table = t;
  return RS_OK;
}

rs_status lookup_pool_bwd(rs_table* t, const rs_ctx* ctx, const void* grad_out, float* grad_unique, rs_stream stream) {
  rs_status st = check_ctx(t, ctx);
  if (st != RS_OK) return st;
  if (ctx->n > 0 && (!grad_out || !grad_unique)) return fail(RS_EINVAL, "null gradient");
  const Work w = ctx_work(ctx);
  RS_HIP(launch_bwd(t->dev(), w, ctx->offsets, ctx->n, ctx->bags, ctx->mode, ctx->pad_len, grad_out, grad_unique,
                    nullptr, t->ev(RS_K_BWD_CHUNKS), t->ev(RS_K_BWD_STRADDLE), static_cast<hipStream_t>(stream)));
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
  RS_HIP(launch_bwd(t->dev(), w, ctx->offsets, ctx->n, ctx->bags, ctx->mode, ctx->pad_len, grad_out, nullptr, &o,
                    t->ev(RS_K_BWD_CHUNKS), t->ev(RS_K_BWD_STRADDLE), static_cast<hipStream_t>(stream)));
  return RS_OK;
}

rs_status rs_set_kernel_events(rs_table* t, int32_t kernel, void* start_event, void* stop_event) {
  if (!t || kernel < 0 || kernel >= RS_K_COUNT) return fail(RS_EINVAL, "bad table or kernel id");
  t->kev[kernel][0] = static_cast<hipEvent_t>(start_event);
  t->kev[kernel][1] = static_cast<hipEvent_t>(stop_event);
  return RS_OK;
}

}  // extern "C"

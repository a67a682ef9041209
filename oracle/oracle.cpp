// CPU oracle for the sparse embedding step — TEST INFRASTRUCTURE ONLY.
//
// Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may load
// this library.  The product path never calls it; it shares no code, header,
// table or constant generator with the HIP library.
//
// It is a plain, slow, sequential C++17 restatement of what the RecIS sparse
// component computes (RecIS, "Optimization for Memory Bound": the two-tier
// IDMap + Blocks store and its forward/backward workflow; "Framework
// Components": the Embedding Engine and the sparse Optimizer; "Benchmark of
// Operators": dedup in ids partition, sum/mean reduction, gather, scatter):
//
//   dedup          unique keys in first-occurrence order + inverse index
//   find-or-insert IDMap key -> row; a missing key gets a free row (or the
//                  next new one) and a deterministic initial value derived
//                  from (seed, key)
//   eviction       keys not looked up for more than a given number of calls
//                  leave the table; their rows are reused
//   forward        per bag: sum / mean of its rows, or a padded copy
//   backward       per unique key: sum of the upstream gradients of every
//                  occurrence (scaled by 1/len for mean)
//   ids partition  dedup + split of the distinct keys by owner shard
//   bucketize/mod  feature transforms fused over many columns
//   optimizer      Adagrad (Duchi et al. 2011), Adam (Kingma & Ba 2015,
//                  Algorithm 1), AdamW (Adam with decoupled weight decay,
//                  Loshchilov & Hutter 2019; the paper names SparseAdamW) or
//                  Adam in the reordered form with epsilon-hat (Kingma & Ba
//                  2015, end of section 2; TensorFlow's Adam), or the
//                  row-wise (one scalar per row) Adagrad / Adam, on the
//                  touched rows only
//
// Sums and optimizer arithmetic are carried in fp64; stored rows and state
// are fp32 (or bf16 rows, rounded to nearest even) because the storage type
// is part of the table's definition.  Every function names the passage it
// follows.  Where the paper is silent the reading taken is stated inline.
//
// Status codes (numeric contract shared with the product ABI by value only):
//   0 OK, 1 EINVAL, 2 ENOMEM, 3 EFULL, 4 EKEY.

#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <unordered_map>
#include <vector>

namespace {

constexpr int ST_OK = 0, ST_EINVAL = 1, ST_EFULL = 3, ST_EKEY = 4;
constexpr int SUM = 0, MEAN = 1, NONE = 2, TAIL = 3;
constexpr int F32 = 0, BF16 = 1;
constexpr int ADAGRAD = 0, ADAM = 1, ADAMW = 2, ADAM_TF = 3, ADAGRAD_RW = 4, ADAM_RW = 5;
constexpr int64_t KEY_EMPTY = std::numeric_limits<int64_t>::min();   // reserved
constexpr int64_t KEY_TOMB = std::numeric_limits<int64_t>::min() + 1; // reserved

// splitmix64 output function (Steele, Lea & Flood, OOPSLA 2014; Vigna's
// public-domain splitmix64): three xor-shift / multiply rounds.
uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// bf16 from fp32, round to nearest, ties to even; NaN -> canonical quiet NaN.
uint16_t bf16_rne(float x) {
  uint32_t b;
  std::memcpy(&b, &x, 4);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu) != 0) return 0x7FC0;
  uint32_t lsb = (b >> 16) & 1u;
  return static_cast<uint16_t>((b + 0x7FFFu + lsb) >> 16);
}

float bf16_to_f32(uint16_t h) {
  uint32_t b = static_cast<uint32_t>(h) << 16;
  float x;
  std::memcpy(&x, &b, 4);
  return x;
}

// Initial value of a new row.  The paper only says a new feature gets a row
// in the KV store; the workload fixes "uniform(lo,hi) from hash(seed,id)".
// Reading taken: element j draws 24 bits from splitmix64 of the key stream
// and maps them exactly onto [0,1) before one fp32 fused multiply-add.
void init_row(uint64_t seed, int64_t key, int dim, float lo, float hi, float* out) {
  const uint64_t z = mix64(static_cast<uint64_t>(key) ^ mix64(seed));
  const float span = hi - lo;  // fp32 subtraction
  for (int j = 0; j < dim; ++j) {
    const uint64_t h = mix64(z + static_cast<uint64_t>(j + 1) * 0x9E3779B97F4A7C15ull);
    const float u = static_cast<float>(h >> 40) * 0x1.0p-24f;  // exact
    out[j] = std::fma(u, span, lo);                              // single rounding
  }
}

struct Table {
  int dim = 0, row_dtype = F32, opt = ADAGRAD;
  float lo = -0.01f, hi = 0.01f;
  uint64_t seed = 0;
  int64_t max_live = -1;  // < 0: unbounded (grow on demand)
  std::unordered_map<int64_t, int64_t> idmap;  // IDMap: key -> row ("offset")
  std::vector<float> w;                        // Blocks, fp32 rows  [live, dim]
  std::vector<uint16_t> wb;                    // Blocks, bf16 rows  [live, dim]
  std::vector<float> s1, s2;                   // Adagrad acc | Adam m, v   [live, dim]
  std::vector<float> sr;                       // row-wise Adagrad acc | row-wise Adam v  [live]
  int64_t t = 0;                               // Adam step count (table-global)
  // Eviction of stale features (Embedding Engine): every lookup call
  // advances the clock; a row remembers its key and the clock of the last
  // call that looked it up.  Freed rows form a stack that new keys take
  // from (top first) before new rows are added.
  int64_t nrows = 0;                           // rows ever allocated
  std::vector<int64_t> row_key;                // key of each row (KEY_EMPTY: free)
  std::vector<uint32_t> row_seen;              // clock of its last lookup
  std::vector<int64_t> free_stack;             // free rows
  uint32_t clock = 0;

  int64_t live() const { return static_cast<int64_t>(idmap.size()); }
  // per-element state vectors, and whether one scalar per row follows them
  int nvec() const { return opt == ADAGRAD ? 1 : opt == ADAGRAD_RW ? 0 : opt == ADAM_RW ? 1 : 2; }
  bool row_scalar() const { return opt == ADAGRAD_RW || opt == ADAM_RW; }
  bool adam_family() const { return opt != ADAGRAD && opt != ADAGRAD_RW; }
  int state_elems() const { return nvec() * dim + (row_scalar() ? 1 : 0); }
  // state element e of row r: [s1 (dim) | s2 (dim) | row scalar], as present
  float get_s(int64_t r, int e) const {
    if (e < nvec() * dim) return e < dim ? s1[r * dim + e] : s2[r * dim + e - dim];
    return sr[r];
  }
  void put_s(int64_t r, int e, float v) {
    if (e < nvec() * dim) (e < dim ? s1[r * dim + e] : s2[r * dim + e - dim]) = v;
    else sr[r] = v;
  }

  float get_w(int64_t r, int j) const {
    return row_dtype == BF16 ? bf16_to_f32(wb[r * dim + j]) : w[r * dim + j];
  }
  void put_w(int64_t r, int j, float v) {
    if (row_dtype == BF16) wb[r * dim + j] = bf16_rne(v);
    else w[r * dim + j] = v;
  }
  int64_t append(int64_t key, const float* vals) {
    const int64_t r = nrows++;
    idmap.emplace(key, r);
    row_key.push_back(key);
    row_seen.push_back(clock);
    for (int j = 0; j < dim; ++j) {
      if (row_dtype == BF16) wb.push_back(bf16_rne(vals[j]));
      else w.push_back(vals[j]);
      if (nvec() >= 1) s1.push_back(0.0f);
      if (nvec() == 2) s2.push_back(0.0f);
    }
    if (row_scalar()) sr.push_back(0.0f);
    return r;
  }
  // A new key's row: the top of the free stack (re-initialised), else a new one.
  int64_t take_row(int64_t key, const float* vals) {
    if (free_stack.empty()) return append(key, vals);
    const int64_t r = free_stack.back();
    free_stack.pop_back();
    idmap.emplace(key, r);
    row_key[r] = key;
    row_seen[r] = clock;
    for (int j = 0; j < dim; ++j) put_w(r, j, vals[j]);
    for (int e = 0; e < state_elems(); ++e) put_s(r, e, 0.0f);
    return r;
  }
};

bool reserved(int64_t k) { return k == KEY_EMPTY || k == KEY_TOMB; }

// Dedup ("ids partition" dedups before sharding; benchmark of operators).
// The paper does not fix the order of the unique set; reading taken: first
// occurrence order, which is canonical and makes the inverse index exact.
int64_t dedup(const int64_t* v, int64_t n, int64_t* uniq, int32_t* inv) {
  std::unordered_map<int64_t, int64_t> seen;
  int64_t U = 0;
  for (int64_t i = 0; i < n; ++i) {
    auto it = seen.find(v[i]);
    if (it == seen.end()) {
      seen.emplace(v[i], U);
      uniq[U] = v[i];
      inv[i] = static_cast<int32_t>(U);
      ++U;
    } else {
      inv[i] = static_cast<int32_t>(it->second);
    }
  }
  return U;
}

// IDMap find-or-insert (two-tier storage: IDMap maps a feature id to an
// offset into Blocks; the KV store is scalable, so a missing id is inserted).
// New rows are numbered in the order the keys are met, and get init_row().
// With a bounded table, keys past the limit are not inserted and get -1.
int find_or_insert(Table* T, const int64_t* keys, int64_t n, int64_t* rows, int64_t* n_new) {
  for (int64_t i = 0; i < n; ++i)
    if (reserved(keys[i])) return ST_EKEY;
  int st = ST_OK;
  int64_t added = 0;
  std::vector<float> tmp(T->dim);
  for (int64_t i = 0; i < n; ++i) {
    auto it = T->idmap.find(keys[i]);
    if (it != T->idmap.end()) {
      rows[i] = it->second;
      T->row_seen[it->second] = T->clock;
      continue;
    }
    if (T->max_live >= 0 && T->live() >= T->max_live) {
      rows[i] = -1;
      st = ST_EFULL;
      continue;
    }
    init_row(T->seed, keys[i], T->dim, T->lo, T->hi, tmp.data());
    rows[i] = T->take_row(keys[i], tmp.data());
    ++added;
  }
  if (n_new) *n_new = added;
  return st;
}

}  // namespace

extern "C" {

uint64_t or_mix64(uint64_t z) { return mix64(z); }
uint16_t or_bf16_rne(float x) { return bf16_rne(x); }
float or_bf16_to_f32(uint16_t h) { return bf16_to_f32(h); }
void or_init_row(uint64_t seed, int64_t key, int dim, float lo, float hi, float* out) {
  init_row(seed, key, dim, lo, hi, out);
}

void* or_create(int dim, int row_dtype, int opt, float lo, float hi, uint64_t seed, int64_t max_live) {
  if (dim <= 0 || (row_dtype != F32 && row_dtype != BF16) || opt < ADAGRAD || opt > ADAM_RW) return nullptr;
  Table* T = new Table;
  T->dim = dim;
  T->row_dtype = row_dtype;
  T->opt = opt;
  T->lo = lo;
  T->hi = hi;
  T->seed = seed;
  T->max_live = max_live;
  return T;
}

void or_destroy(void* h) { delete static_cast<Table*>(h); }
int64_t or_size(void* h) { return static_cast<Table*>(h)->live(); }
int64_t or_step_count(void* h) { return static_cast<Table*>(h)->t; }
void or_set_step_count(void* h, int64_t t) { static_cast<Table*>(h)->t = t; }

// Returns U, or -ST_EKEY when a reserved key is present.
int64_t or_dedup(const int64_t* values, int64_t n, int64_t* unique_out, int32_t* inverse_out) {
  for (int64_t i = 0; i < n; ++i)
    if (reserved(values[i])) return -ST_EKEY;
  return dedup(values, n, unique_out, inverse_out);
}

// Ids partition ("Ids Partition" in Benchmark of Operators; "Request Merging
// & Sharding" in Load Balancing): the batch's ids are deduplicated and split
// by the shard that owns them, so that each shard can be sent its own ids.
// Reading taken (the paper names no owner function): the owner of key k among
// G shards is mix64(uint64(k) XOR owner_seed) mod G; the output lists the
// distinct keys shard by shard (shard 0 first), each shard's keys in the
// order of their first occurrence in the batch.  shard_offsets[s] is where
// shard s starts (shard_offsets[G] = U); inverse_out[i] is the output
// position of values[i].  A reserved key (INT64_MIN, INT64_MIN+1) takes no
// part: its inverse is -1 and *n_rejected counts it.
// Returns U, or -ST_EINVAL for G < 1.
int64_t or_ids_partition(const int64_t* values, int64_t n, int32_t nshards, uint64_t owner_seed, int64_t* keys_out,
                         int64_t* shard_offsets, int32_t* inverse_out, int64_t* n_rejected) {
  if (nshards < 1 || n < 0) return -ST_EINVAL;
  // 1. distinct keys in first-occurrence order
  std::unordered_map<int64_t, int64_t> first_index;  // key -> index in `order`
  std::vector<int64_t> order;
  int64_t rejected = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (reserved(values[i])) {
      ++rejected;
      continue;
    }
    if (first_index.find(values[i]) == first_index.end()) {
      first_index.emplace(values[i], static_cast<int64_t>(order.size()));
      order.push_back(values[i]);
    }
  }
  // 2. shard by shard, that shard's keys in first-occurrence order
  std::unordered_map<int64_t, int64_t> out_pos;
  int64_t U = 0;
  for (int32_t s = 0; s < nshards; ++s) {
    shard_offsets[s] = U;
    for (int64_t k : order) {
      const uint64_t owner = mix64(static_cast<uint64_t>(k) ^ owner_seed) % static_cast<uint64_t>(nshards);
      if (owner != static_cast<uint64_t>(s)) continue;
      keys_out[U] = k;
      out_pos.emplace(k, U);
      ++U;
    }
  }
  shard_offsets[nshards] = U;
  // 3. each id's position in the output
  for (int64_t i = 0; i < n; ++i)
    inverse_out[i] = reserved(values[i]) ? -1 : static_cast<int32_t>(out_pos.at(values[i]));
  if (n_rejected) *n_rejected = rejected;
  return U;
}

// Bucketize, fused over columns ("Bucketize and Mod" in Benchmark of
// Operators; the Feature Engine turns a float feature such as a price into
// an id by its bucket).  Column c holds values[col_off[c] .. col_off[c+1])
// and its nondecreasing boundaries bnd[bnd_off[c] .. bnd_off[c+1]).
// Reading taken (the paper names the operator only): TensorFlow's Bucketize,
// an upper-bound search: bucket = the index of the first boundary b with
// x < b, or the number of boundaries if there is none (so boundaries[k-1] <=
// x < boundaries[k] gives k); a NaN is below no boundary and lands in the
// last bucket.
// Returns 0, or -ST_EINVAL for bad offsets.
int or_bucketize(const float* values, const int64_t* col_off, int32_t ncols, const float* bnd,
                 const int64_t* bnd_off, int64_t* out) {
  if (ncols < 0 || col_off[0] != 0 || bnd_off[0] != 0) return -ST_EINVAL;
  for (int32_t c = 0; c < ncols; ++c) {
    if (col_off[c + 1] < col_off[c] || bnd_off[c + 1] < bnd_off[c]) return -ST_EINVAL;
    for (int64_t i = col_off[c]; i < col_off[c + 1]; ++i) {
      int64_t k = 0;  // first boundary above the value
      while (bnd_off[c] + k < bnd_off[c + 1] && !(values[i] < bnd[bnd_off[c] + k])) ++k;
      out[i] = k;
    }
  }
  return 0;
}

// Mod, fused over columns (same passage): column c's ids map to x mod m_c
// with m_c > 0.  Reading taken: the floor modulus (result in [0, m_c), also
// for a negative id), so the result is a valid bucket id.
int or_mod(const int64_t* values, const int64_t* col_off, int32_t ncols, const int64_t* moduli, int64_t* out) {
  if (ncols < 0 || col_off[0] != 0) return -ST_EINVAL;
  for (int32_t c = 0; c < ncols; ++c) {
    if (col_off[c + 1] < col_off[c] || moduli[c] <= 0) return -ST_EINVAL;
    for (int64_t i = col_off[c]; i < col_off[c + 1]; ++i) {
      int64_t r = values[i] % moduli[c];
      if (r < 0) r += moduli[c];
      out[i] = r;
    }
  }
  return 0;
}

int or_find_or_insert(void* h, const int64_t* keys, int64_t n, int64_t* rows_out, int64_t* n_inserted) {
  static_cast<Table*>(h)->clock += 1;  // one lookup call
  return find_or_insert(static_cast<Table*>(h), keys, n, rows_out, n_inserted);
}

// Evict the stale features: every key whose age (clock now minus the clock
// of its last lookup, modulo 2^32) exceeds max_age leaves the IDMap; its row
// is pushed on the free stack (rows in ascending order).  Returns the count.
int64_t or_evict(void* h, uint32_t max_age) {
  Table* T = static_cast<Table*>(h);
  int64_t count = 0;
  for (int64_t r = 0; r < T->nrows; ++r) {
    if (T->row_key[r] == KEY_EMPTY) continue;
    if (static_cast<uint32_t>(T->clock - T->row_seen[r]) <= max_age) continue;
    T->idmap.erase(T->row_key[r]);
    T->row_key[r] = KEY_EMPTY;
    T->free_stack.push_back(r);
    ++count;
  }
  return count;
}

// Compaction of the Blocks after eviction.  The paper sizes its Blocks
// flexibly (they grow by appending memory blocks) and evicts stale
// features, but gives no procedure for giving rows back; the reading taken:
// with L live keys, each row r >= L that holds a key moves into a free row
// below L -- the k-th such row in ascending order into the k-th free row
// below L in ascending order -- with its values, optimizer state and
// last-lookup clock, and the IDMap follows it.  Afterwards rows 0 .. L-1
// hold every live key, no row is free, and L rows are allocated, so memory
// past row L can be released.  Returns the number of rows moved.
int64_t or_compact(void* h) {
  Table* T = static_cast<Table*>(h);
  const int64_t L = T->live();
  std::vector<int64_t> holes, movers;
  for (int64_t r = 0; r < L && r < T->nrows; ++r)
    if (T->row_key[r] == KEY_EMPTY) holes.push_back(r);
  for (int64_t r = L; r < T->nrows; ++r)
    if (T->row_key[r] != KEY_EMPTY) movers.push_back(r);
  if (holes.size() != movers.size()) return -1;  // cannot happen: both count the keys missing below L
  for (size_t k = 0; k < movers.size(); ++k) {
    const int64_t src = movers[k], dst = holes[k];
    for (int j = 0; j < T->dim; ++j) {
      if (T->row_dtype == BF16) T->wb[dst * T->dim + j] = T->wb[src * T->dim + j];
      else T->w[dst * T->dim + j] = T->w[src * T->dim + j];
    }
    for (int e = 0; e < T->state_elems(); ++e) T->put_s(dst, e, T->get_s(src, e));
    T->row_key[dst] = T->row_key[src];
    T->row_seen[dst] = T->row_seen[src];
    T->idmap[T->row_key[src]] = dst;
  }
  // rows L and beyond are gone
  T->nrows = L;
  T->row_key.resize(L);
  T->row_seen.resize(L);
  if (T->row_dtype == BF16) T->wb.resize(L * T->dim);
  else T->w.resize(L * T->dim);
  if (T->nvec() >= 1) T->s1.resize(L * T->dim);
  if (T->nvec() == 2) T->s2.resize(L * T->dim);
  if (T->row_scalar()) T->sr.resize(L);
  T->free_stack.clear();
  return static_cast<int64_t>(movers.size());
}

int64_t or_rows_allocated(void* h) { return static_cast<Table*>(h)->nrows; }
uint32_t or_clock(void* h) { return static_cast<Table*>(h)->clock; }

// Row contents by key (w as fp32 values; state_elems() state floats per key:
// [acc] / [m | v] per element, or the row-wise [acc] / [m (dim) | v]).
// Returns the number of keys found; absent keys leave their output untouched.
int64_t or_read_rows(void* h, const int64_t* keys, int64_t n, float* w_out, float* state_out) {
  Table* T = static_cast<Table*>(h);
  const int D = T->dim, S = T->state_elems();
  int64_t found = 0;
  for (int64_t i = 0; i < n; ++i) {
    auto it = T->idmap.find(keys[i]);
    if (it == T->idmap.end()) continue;
    ++found;
    const int64_t r = it->second;
    for (int j = 0; j < D; ++j)
      if (w_out) w_out[i * D + j] = T->get_w(r, j);
    for (int e = 0; e < S; ++e)
      if (state_out) state_out[i * S + e] = T->get_s(r, e);
  }
  return found;
}

// Overwrite (or create) rows by key — used by stage-wise tests to start the
// oracle from a given table state.  w values are rounded to the row dtype.
void or_write_rows(void* h, const int64_t* keys, int64_t n, const float* w_in, const float* state_in) {
  Table* T = static_cast<Table*>(h);
  const int D = T->dim, S = T->state_elems();
  std::vector<float> zero(D, 0.0f);
  for (int64_t i = 0; i < n; ++i) {
    auto it = T->idmap.find(keys[i]);
    int64_t r = (it == T->idmap.end()) ? T->append(keys[i], zero.data()) : it->second;
    for (int j = 0; j < D; ++j) T->put_w(r, j, w_in[i * D + j]);
    for (int e = 0; e < S; ++e) T->put_s(r, e, state_in ? state_in[i * S + e] : 0.0f);
  }
}

int64_t or_export(void* h, int64_t* keys, int64_t* rows, int64_t cap) {
  Table* T = static_cast<Table*>(h);
  int64_t i = 0;
  for (const auto& kv : T->idmap) {
    if (i < cap) {
      keys[i] = kv.first;
      rows[i] = kv.second;
    }
    ++i;
  }
  return i;
}

// Forward (workflow, forward pass: one IDMap lookup per id, then the row at
// that offset; pooling modes sum / mean / padded copy from the reduction
// operators).  Input is CSR: values[n], offsets[bags+1].
//   SUM : out[g]       = sum of rows of bag g                 (fp64)
//   MEAN: out[g]       = that sum / len(g); an empty bag gives 0
//   NONE: out[g][t]    = row of the t-th id of bag g for t < min(len, L), else 0;
//         mask[g][t]   = t < len
//   TAIL: the same with the last min(len, L) ids of the bag: out[g][t] = row of
//         id skip + t, skip = max(len - L, 0) (the sequence tile of the
//         Reduction Operations, concatenating a sequence's most recent rows)
// Dedup and find-or-insert run first (new keys are inserted during the
// forward, so new rows are initialised before use).  A row of -1 (a failed
// insert in a bounded table) contributes a zero vector.
int or_forward(void* h, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags,
               int mode, int64_t pad_len, double* out, uint8_t* mask, int64_t* unique_out,
               int32_t* inverse_out, int64_t* rows_out, int64_t* U_out, int64_t* n_new_out) {
  Table* T = static_cast<Table*>(h);
  if (n < 0 || bags < 0 || offsets[0] != 0 || offsets[bags] != n) return ST_EINVAL;
  for (int64_t g = 0; g < bags; ++g)
    if (offsets[g + 1] < offsets[g]) return ST_EINVAL;
  if ((mode == NONE || mode == TAIL) && pad_len <= 0) return ST_EINVAL;
  const int64_t U = or_dedup(values, n, unique_out, inverse_out);
  if (U < 0) return ST_EKEY;
  int64_t nn = 0;
  T->clock += 1;  // one lookup call
  int st = find_or_insert(T, unique_out, U, rows_out, &nn);
  *U_out = U;
  *n_new_out = nn;
  const int D = T->dim;
  for (int64_t g = 0; g < bags; ++g) {
    const int64_t b = offsets[g], e = offsets[g + 1], len = e - b;
    if (mode == NONE || mode == TAIL) {
      const int64_t skip = mode == TAIL && len > pad_len ? len - pad_len : 0;
      for (int64_t t = 0; t < pad_len; ++t) {
        double* o = out + (g * pad_len + t) * D;
        mask[g * pad_len + t] = static_cast<uint8_t>(t < len);
        const int64_t r = t < len ? rows_out[inverse_out[b + skip + t]] : -1;
        for (int j = 0; j < D; ++j) o[j] = r >= 0 ? static_cast<double>(T->get_w(r, j)) : 0.0;
      }
      continue;
    }
    double* o = out + g * D;
    for (int j = 0; j < D; ++j) o[j] = 0.0;
    for (int64_t i = b; i < e; ++i) {
      const int64_t r = rows_out[inverse_out[i]];
      if (r < 0) continue;
      for (int j = 0; j < D; ++j) o[j] += static_cast<double>(T->get_w(r, j));
    }
    if (mode == MEAN && len > 0)
      for (int j = 0; j < D; ++j) o[j] /= static_cast<double>(len);
  }
  return st;
}

// Backward (workflow, backward update: gradients are aggregated per
// retained forward offset).  grad_unique[u] = sum over occurrences i of key u
// of scale(g(i)) * grad[g(i)], scale = 1 (sum) or 1/len (mean); padded mode
// sums grad[g][t] over the positions t < min(len, L) holding key u (tail
// mode: id skip + t holds slot t).  Masked positions are never read.  Sums
// in fp64.
int or_backward(const int64_t* offsets, int64_t bags, const int32_t* inverse, int64_t U, int dim,
                int mode, int64_t pad_len, const float* grad, double* grad_unique) {
  for (int64_t k = 0; k < U * dim; ++k) grad_unique[k] = 0.0;
  for (int64_t g = 0; g < bags; ++g) {
    const int64_t b = offsets[g], e = offsets[g + 1], len = e - b;
    const int64_t skip = mode == TAIL && len > pad_len ? len - pad_len : 0;
    for (int64_t i = b; i < e; ++i) {
      const int64_t u = inverse[i];
      if (u < 0) continue;
      double* gu = grad_unique + u * dim;
      if (mode == NONE || mode == TAIL) {
        const int64_t t = i - b - skip;
        if (t < 0 || t >= pad_len) continue;
        const float* gr = grad + (g * pad_len + t) * dim;
        for (int j = 0; j < dim; ++j) gu[j] += static_cast<double>(gr[j]);
      } else {
        const float* gr = grad + g * dim;
        const double sc = mode == MEAN ? 1.0 / static_cast<double>(len) : 1.0;
        for (int j = 0; j < dim; ++j) gu[j] += sc * static_cast<double>(gr[j]);
      }
    }
  }
  return ST_OK;
}

// Row-sparse optimizer (SparseAdam-style: only the rows touched this step
// are read and written; untouched rows and their state stay as they are).
//   Adagrad: acc += g^2;  w -= lr * g / (sqrt(acc) + eps)          (initial acc 0)
//   Adam:    t += 1 once per call (table-global step);
//            m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;
//            w -= lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)
//   AdamW:   the Adam step applied to w - lr * wd * w (decoupled decay of
//            the touched row, then the moment update and step)
//   Adam (epsilon-hat form): the same moments; lr_t = lr * sqrt(1-b2^t) / (1-b1^t);
//            w -= lr_t * m / (sqrt(v) + eps)
//   Row-wise state (one scalar per row instead of one per element; the
//   memory-saving form of embedding-table optimizers, as in FBGEMM), with
//   ms = mean over the row of g^2:
//   Row-wise Adagrad: acc += ms;  w -= lr * g / (sqrt(acc) + eps)
//   Row-wise Adam:    m per element as in Adam; v = b2 v + (1-b2) ms per
//            row;  w -= lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)
// Arithmetic in fp64 from the stored fp32 state; results stored as fp32
// state and fp32 (or bf16, via fp32 then round-to-nearest-even) rows.
// rows[u] < 0 is skipped.  grad is fp32 [U, dim].
int or_optimizer(void* h, const int64_t* rows, int64_t U, const float* grad, double lr, double eps,
                 double beta1, double beta2, double weight_decay) {
  Table* T = static_cast<Table*>(h);
  const int D = T->dim;
  double bc1 = 1.0, bc2 = 1.0;
  if (T->adam_family()) {
    T->t += 1;
    bc1 = 1.0 - std::pow(beta1, static_cast<double>(T->t));
    bc2 = 1.0 - std::pow(beta2, static_cast<double>(T->t));
  }
  const double lr_t = lr * std::sqrt(bc2) / bc1;
  for (int64_t u = 0; u < U; ++u) {
    const int64_t r = rows[u];
    if (r < 0) continue;
    if (T->row_scalar()) {
      // one accumulator per row from the mean of the squared gradient
      double ms = 0.0;
      for (int j = 0; j < D; ++j) {
        const double g = static_cast<double>(grad[u * D + j]);
        ms += g * g;
      }
      ms /= static_cast<double>(D);
      if (T->opt == ADAGRAD_RW) {
        const double acc = static_cast<double>(T->sr[r]) + ms;
        const double step = lr / (std::sqrt(acc) + eps);
        for (int j = 0; j < D; ++j)
          T->put_w(r, j, static_cast<float>(static_cast<double>(T->get_w(r, j)) -
                                            step * static_cast<double>(grad[u * D + j])));
        T->sr[r] = static_cast<float>(acc);
      } else {
        const double v = beta2 * static_cast<double>(T->sr[r]) + (1.0 - beta2) * ms;
        const double den = std::sqrt(v / bc2) + eps;
        for (int j = 0; j < D; ++j) {
          const double g = static_cast<double>(grad[u * D + j]);
          const double m = beta1 * static_cast<double>(T->s1[r * D + j]) + (1.0 - beta1) * g;
          T->put_w(r, j, static_cast<float>(static_cast<double>(T->get_w(r, j)) - lr * (m / bc1) / den));
          T->s1[r * D + j] = static_cast<float>(m);
        }
        T->sr[r] = static_cast<float>(v);
      }
      continue;
    }
    for (int j = 0; j < D; ++j) {
      const double g = static_cast<double>(grad[u * D + j]);
      double w = static_cast<double>(T->get_w(r, j));
      if (T->opt == ADAGRAD) {
        const double acc = static_cast<double>(T->s1[r * D + j]) + g * g;
        w -= lr * g / (std::sqrt(acc) + eps);
        T->s1[r * D + j] = static_cast<float>(acc);
      } else {
        const double m = beta1 * static_cast<double>(T->s1[r * D + j]) + (1.0 - beta1) * g;
        const double v = beta2 * static_cast<double>(T->s2[r * D + j]) + (1.0 - beta2) * g * g;
        if (T->opt == ADAM_TF) {
          w -= lr_t * m / (std::sqrt(v) + eps);
        } else {
          if (T->opt == ADAMW) w -= lr * weight_decay * w;
          w -= lr * (m / bc1) / (std::sqrt(v / bc2) + eps);
        }
        T->s1[r * D + j] = static_cast<float>(m);
        T->s2[r * D + j] = static_cast<float>(v);
      }
      T->put_w(r, j, static_cast<float>(w));
    }
  }
  return ST_OK;
}

// One training step: forward (with inserts), backward, gradients rounded to
// fp32 (the method's grad_unique dtype), then the optimizer.
int or_step(void* h, const int64_t* values, const int64_t* offsets, int64_t n, int64_t bags, int mode,
            int64_t pad_len, const float* grad, double lr, double eps, double beta1, double beta2,
            double weight_decay, double* out, uint8_t* mask, int64_t* U_out, int64_t* n_new_out) {
  Table* T = static_cast<Table*>(h);
  std::vector<int64_t> uniq(static_cast<size_t>(n > 0 ? n : 1)), rows(static_cast<size_t>(n > 0 ? n : 1));
  std::vector<int32_t> inv(static_cast<size_t>(n > 0 ? n : 1));
  int st = or_forward(h, values, offsets, n, bags, mode, pad_len, out, mask, uniq.data(), inv.data(),
                      rows.data(), U_out, n_new_out);
  if (st != ST_OK && st != ST_EFULL) return st;
  const int64_t U = *U_out;
  const int D = T->dim;
  std::vector<double> gu(static_cast<size_t>(U * D > 0 ? U * D : 1));
  or_backward(offsets, bags, inv.data(), U, D, mode, pad_len, grad, gu.data());
  std::vector<float> g32(gu.size());
  for (size_t k = 0; k < gu.size(); ++k) g32[k] = static_cast<float>(gu[k]);
  or_optimizer(h, rows.data(), U, g32.data(), lr, eps, beta1, beta2, weight_decay);
  return st;
}

}  // extern "C"

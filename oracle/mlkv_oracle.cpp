// CPU oracle for the batched embedding get / put_grad path.
//
// TEST INFRASTRUCTURE ONLY. This file is the plain, slow, single-threaded
// definition that the GPU library is checked against. Only the test suite,
// the smoke check and the benchmark's CPU-baseline leg may load it. It shares
// no code, header, constant table or helper with the GPU library.
//
// What it computes (MLKV, arXiv 2504.01506):
//   * Open(model_id, dim, staleness_bound) creates a table of `dim`-wide
//     embedding rows (Sec. III-A, "Interfaces Summary"). Here: one table
//     with a capacity, and either no staleness bound or a bound s >= 0 kept
//     with the per-key counts of R8 (Sec. III-C1).
//   * Get(keys) returns the embedding vector of each key (Sec. III-A). A key
//     that is not present is inserted with a seeded initial row first.
//   * Rmw (Sec. III-B, workflow step 8) with the modify function
//     "sum the gradients of duplicate keys, then one row-wise Adagrad step".
//     The update has the form of the paper's embedding update (Sec. II-A,
//     w_{t+1} = w_t - gamma * grad) with an Adagrad-scaled gradient.
//
// Readings of points the paper leaves open:
//   R1  rows are dense in [0, size); within one call the distinct keys that
//       are missing receive consecutive rows in ascending key order.
//   R2  the initial value of element c of key k is a fixed function of
//       (seed, k, c) only (SplitMix64 finaliser, Steele, Lea & Flood 2014).
//   R3  duplicate keys in one put are summed (fp64, ascending position,
//       rounded once to fp32), then ONE Adagrad step is applied per key.
//   R4  row-wise Adagrad: m = mean_c(g_c^2) computed in fp64 and rounded to
//       fp32; G' = G + m; den = sqrt(G') + eps; w_c -= lr * (g_c / den);
//       all fp32 operations separate (no fused multiply-add).
//   R5  a call that would exceed the capacity fails as a whole (EFULL) and
//       leaves the table unchanged; a reserved key (all ones) is EINVAL.
//   R6  Put(keys, values) (Sec. III-A, an upsert) applied as one batch: the
//       value at the last position of a key wins; missing keys are inserted
//       as in R1; the Adagrad accumulator of an existing key is kept, a new
//       key's is 0.
//   R7  the SGD variant of the Rmw applies the paper's update form itself
//       (Sec. II-A): duplicate gradients summed as in R3, then
//       w_c -= lr * g_c (separate fp32 operations); accumulators untouched.
//   R8  bounded staleness (Sec. III-C1, the per-record vector clock): a table
//       opened with a staleness bound s >= 0 keeps a count c_k per key, the
//       gets served on k not yet matched by a put. A get call serves an
//       already present key only while c_k <= s (the paper's strict "below
//       the bound" could never serve anything at s = 0, its bulk-synchronous
//       setting, so the test is read as <=) and then raises c_k by one; a key
//       that fails the test is blocked: its positions of `out` are left as
//       they are, c_k is unchanged, and the call reports the positions. The
//       count moves once per call and key, however often the key occurs in
//       the call. A key that the get inserts is served with c_k = 1. Every
//       put call (any modify function) lowers c_k of each distinct key by one,
//       never below 0 (the paper's Put only reduces the staleness); a key a
//       put inserts starts at 0. Without a bound nothing is counted and every
//       get is served (the asynchronous end, bound = infinity). Waiting is
//       left to the caller, which repeats a blocked get after the puts it
//       waits for.
//   R9  Lookahead(keys) (Sec. III-A; look-ahead prefetching, Sec. III-C2)
//       with the whole table in memory: the keys are made resident ahead of
//       the gets that will read them, i.e. the missing ones are inserted as
//       in R1 with their initial rows; nothing is returned, and no staleness
//       count changes (a prefetched record keeps its staleness; a new one
//       starts at 0).
//
// Storage is deliberately naive: std::unordered_map for key -> row, a sorted
// array for a bulk prefill (identical result to inserting the same ascending
// keys through get), and rows are materialised only when first written
// (an untouched row equals its initial value by definition).

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <unordered_map>
#include <vector>

namespace {

constexpr int kOk = 0;
constexpr int kEinval = -1;
constexpr int kEfull = -2;
constexpr uint64_t kReservedKey = ~0ull;

// SplitMix64 output function ("mix64", variant 13 constants), from Steele,
// Lea & Flood, "Fast splittable pseudorandom number generators" (OOPSLA 2014).
uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// R2: initial value of element c of `key`.
float init_value(uint64_t seed, uint64_t key, int32_t c) {
  const uint64_t h = splitmix64_mix(splitmix64_mix(key ^ seed) +
                                    (uint64_t)(uint32_t)c * 0x9E3779B97F4A7C15ull);
  const int32_t t = (int32_t)(h >> 40) - (1 << 23);   // in [-2^23, 2^23)
  const float scale = 0.01f * 0x1p-23f;               // exact power-of-two scaling
  return (float)t * scale;
}

struct Table {
  int32_t dim;
  int64_t capacity;
  uint64_t seed;
  int64_t size = 0;
  // rows [0, prefill_n) belong to the keys of a bulk prefill, in ascending order
  std::vector<uint64_t> row_key;                 // key of every row in [0, size)
  int64_t prefill_n = 0;
  std::unordered_map<uint64_t, uint32_t> map;    // keys inserted one call at a time
  std::unordered_map<uint32_t, size_t> stored;   // row -> offset in `store` once written
  std::vector<float> store;
  std::unordered_map<uint32_t, float> accum;     // row -> Adagrad accumulator G (0 if absent)
  int64_t bound = -1;                            // staleness bound (R8); -1: not tracked
  std::unordered_map<uint32_t, uint32_t> stale;  // row -> c_k (0 if absent), when tracked
};

// R8, put side: one completed update for every distinct row of the call.
void put_done(Table& t, const std::vector<uint32_t>& rows) {
  if (t.bound < 0) return;
  std::vector<uint32_t> u(rows);
  std::sort(u.begin(), u.end());
  u.erase(std::unique(u.begin(), u.end()), u.end());
  for (uint32_t r : u) {
    auto it = t.stale.find(r);
    if (it != t.stale.end() && it->second > 0) it->second -= 1;
  }
}

bool find_row(const Table& t, uint64_t key, uint32_t* row) {
  if (t.prefill_n > 0) {
    auto first = t.row_key.begin();
    auto last = t.row_key.begin() + t.prefill_n;
    auto it = std::lower_bound(first, last, key);
    if (it != last && *it == key) {
      *row = (uint32_t)(it - first);
      return true;
    }
  }
  auto it = t.map.find(key);
  if (it == t.map.end()) return false;
  *row = it->second;
  return true;
}

float read_elem(const Table& t, uint32_t row, int32_t c) {
  auto it = t.stored.find(row);
  if (it != t.stored.end()) return t.store[it->second + (size_t)c];
  return init_value(t.seed, t.row_key[row], c);
}

float* writable_row(Table& t, uint32_t row) {
  auto it = t.stored.find(row);
  if (it == t.stored.end()) {
    const size_t off = t.store.size();
    t.store.resize(off + (size_t)t.dim);
    for (int32_t c = 0; c < t.dim; ++c) t.store[off + (size_t)c] = init_value(t.seed, t.row_key[row], c);
    it = t.stored.emplace(row, off).first;
  }
  return t.store.data() + it->second;
}

int check_keys(const uint64_t* keys, int64_t n) {
  if (n < 0 || n > 0x7FFFFFFFll) return kEinval;
  if (n > 0 && keys == nullptr) return kEinval;
  for (int64_t i = 0; i < n; ++i)
    if (keys[i] == kReservedKey) return kEinval;
  return kOk;
}

// R1/R5: map every key to its row, inserting the missing ones.
int resolve(Table& t, const uint64_t* keys, int64_t n, std::vector<uint32_t>* rows) {
  std::vector<uint64_t> missing;
  for (int64_t i = 0; i < n; ++i) {
    uint32_t r;
    if (!find_row(t, keys[i], &r)) missing.push_back(keys[i]);
  }
  std::sort(missing.begin(), missing.end());
  missing.erase(std::unique(missing.begin(), missing.end()), missing.end());
  if (t.size + (int64_t)missing.size() > t.capacity) return kEfull;
  for (size_t j = 0; j < missing.size(); ++j) {
    const uint32_t row = (uint32_t)(t.size + (int64_t)j);
    t.map.emplace(missing[j], row);
    t.row_key.push_back(missing[j]);
  }
  t.size += (int64_t)missing.size();
  if (rows) {
    rows->resize((size_t)n);
    for (int64_t i = 0; i < n; ++i) find_row(t, keys[i], &(*rows)[(size_t)i]);
  }
  return kOk;
}

}  // namespace

extern "C" {

typedef struct oracle_table oracle_table;

int oracle_abi_version(void) { return 1; }

oracle_table* oracle_open(int32_t dim, int64_t capacity, uint64_t seed) {
  if (dim <= 0 || capacity < 1 || capacity > 0xFFFFFFFEll) return nullptr;
  Table* t = new Table();
  t->dim = dim;
  t->capacity = capacity;
  t->seed = seed;
  return reinterpret_cast<oracle_table*>(t);
}

// Open with a staleness bound s >= 0 (R8; Sec. III-C1: s = 0 is bulk-synchronous).
oracle_table* oracle_open_bounded(int32_t dim, int64_t capacity, uint64_t seed, int64_t bound) {
  if (bound < 0) return nullptr;
  oracle_table* h = oracle_open(dim, capacity, seed);
  if (h) reinterpret_cast<Table*>(h)->bound = bound;
  return h;
}

void oracle_close(oracle_table* h) { delete reinterpret_cast<Table*>(h); }

int64_t oracle_size(oracle_table* h) { return reinterpret_cast<Table*>(h)->size; }

float oracle_init_value(uint64_t seed, uint64_t key, int32_t c) { return init_value(seed, key, c); }

uint64_t oracle_mix64(uint64_t z) { return splitmix64_mix(z); }

// Bulk prefill of an EMPTY table with strictly ascending keys: identical in
// effect to oracle_get(keys, n, NULL) (every key is missing, so row = rank),
// but held as a sorted array instead of n hash-map entries.
int oracle_prefill_sorted(oracle_table* h, const uint64_t* keys, int64_t n) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (check_keys(keys, n) != kOk) return kEinval;
  if (t.size != 0) return kEinval;
  for (int64_t i = 1; i < n; ++i)
    if (!(keys[i - 1] < keys[i])) return kEinval;
  if (n > t.capacity) return kEfull;
  t.row_key.assign(keys, keys + n);
  t.prefill_n = n;
  t.size = n;
  return kOk;
}

// Get (Sec. III-A): out[i][c] = W[row(keys[i])][c]; `out` may be NULL (insert only).
int oracle_get(oracle_table* h, const uint64_t* keys, int64_t n, float* out) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (t.bound >= 0) return kEinval;  // a bounded table reports blocked keys: oracle_get_bounded
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  std::vector<uint32_t> rows;
  rc = resolve(t, keys, n, &rows);
  if (rc != kOk) return rc;
  if (out) {
    for (int64_t i = 0; i < n; ++i)
      for (int32_t c = 0; c < t.dim; ++c)
        out[i * t.dim + c] = read_elem(t, rows[(size_t)i], c);
  }
  return kOk;
}

// Get under the staleness bound (R8): each distinct key of the call is served
// if its count before the call is at most the bound (a key the call inserts
// has count 0), and a served key's count then grows by one. blocked[i] = 1
// where keys[i] is blocked (out row i left as it is), else 0 and out row i is
// the key's row as in oracle_get.
int oracle_get_bounded(oracle_table* h, const uint64_t* keys, int64_t n, float* out, uint8_t* blocked) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (t.bound < 0) return kEinval;
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  if (n > 0 && blocked == nullptr) return kEinval;
  std::vector<uint32_t> rows;
  rc = resolve(t, keys, n, &rows);
  if (rc != kOk) return rc;
  std::map<uint32_t, bool> served;  // verdict of every distinct row, on its count before the call
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t r = rows[(size_t)i];
    if (served.count(r)) continue;
    auto it = t.stale.find(r);
    const uint32_t c = it == t.stale.end() ? 0u : it->second;
    served[r] = (int64_t)c <= t.bound;
  }
  for (const auto& kv : served)
    if (kv.second) t.stale[kv.first] += 1;
  for (int64_t i = 0; i < n; ++i) {
    const bool ok = served[rows[(size_t)i]];
    blocked[i] = ok ? 0 : 1;
    if (ok && out)
      for (int32_t c = 0; c < t.dim; ++c) out[i * t.dim + c] = read_elem(t, rows[(size_t)i], c);
  }
  return kOk;
}

// Lookahead (R9): insert the missing keys (R1, R5); no output, no counts.
int oracle_lookahead(oracle_table* h, const uint64_t* keys, int64_t n) {
  Table& t = *reinterpret_cast<Table*>(h);
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  return resolve(t, keys, n, nullptr);
}

// Rmw with "sum duplicates, then row-wise Adagrad" (R3, R4).
int oracle_put_grad(oracle_table* h, const uint64_t* keys, const float* grads, int64_t n,
                    float lr, float eps) {
  Table& t = *reinterpret_cast<Table*>(h);
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  if (n > 0 && grads == nullptr) return kEinval;
  if (!std::isfinite(lr) || !std::isfinite(eps) || eps < 0.0f) return kEinval;
  std::vector<uint32_t> rows;
  rc = resolve(t, keys, n, &rows);
  if (rc != kOk) return rc;

  // positions of every distinct row, ascending
  std::map<uint32_t, std::vector<int64_t>> groups;
  for (int64_t i = 0; i < n; ++i) groups[rows[(size_t)i]].push_back(i);

  const int32_t D = t.dim;
  std::vector<float> g((size_t)D);
  for (const auto& kv : groups) {
    const uint32_t u = kv.first;
    for (int32_t c = 0; c < D; ++c) {
      double s = 0.0;
      for (int64_t i : kv.second) s += (double)grads[i * D + c];
      g[(size_t)c] = (float)s;
    }
    double sq = 0.0;
    for (int32_t c = 0; c < D; ++c) sq += (double)g[(size_t)c] * (double)g[(size_t)c];
    const float m = (float)(sq / (double)D);
    float G = 0.0f;
    auto it = t.accum.find(u);
    if (it != t.accum.end()) G = it->second;
    const float Gn = G + m;
    const float den = std::sqrt(Gn) + eps;
    float* w = writable_row(t, u);
    for (int32_t c = 0; c < D; ++c) {
      const float q = g[(size_t)c] / den;
      const float p = lr * q;
      w[c] = w[c] - p;
    }
    t.accum[u] = Gn;
  }
  put_done(t, rows);
  return kOk;
}

// Put (Sec. III-A) as a batch upsert (R6): W[row(keys[i])] = values[i] for the
// last position i of every distinct key.
int oracle_put(oracle_table* h, const uint64_t* keys, const float* values, int64_t n) {
  Table& t = *reinterpret_cast<Table*>(h);
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  if (n > 0 && values == nullptr) return kEinval;
  std::vector<uint32_t> rows;
  rc = resolve(t, keys, n, &rows);
  if (rc != kOk) return rc;
  std::map<uint32_t, int64_t> last;  // row -> its last position
  for (int64_t i = 0; i < n; ++i) last[rows[(size_t)i]] = i;
  for (const auto& kv : last) {
    float* w = writable_row(t, kv.first);
    for (int32_t c = 0; c < t.dim; ++c) w[c] = values[kv.second * t.dim + c];
  }
  put_done(t, rows);
  return kOk;
}

// Rmw with "sum duplicates, then one plain SGD step" (R7).
int oracle_put_grad_sgd(oracle_table* h, const uint64_t* keys, const float* grads, int64_t n, float lr) {
  Table& t = *reinterpret_cast<Table*>(h);
  int rc = check_keys(keys, n);
  if (rc != kOk) return rc;
  if (n > 0 && grads == nullptr) return kEinval;
  if (!std::isfinite(lr)) return kEinval;
  std::vector<uint32_t> rows;
  rc = resolve(t, keys, n, &rows);
  if (rc != kOk) return rc;
  std::map<uint32_t, std::vector<int64_t>> groups;
  for (int64_t i = 0; i < n; ++i) groups[rows[(size_t)i]].push_back(i);
  const int32_t D = t.dim;
  for (const auto& kv : groups) {
    float* w = writable_row(t, kv.first);
    for (int32_t c = 0; c < D; ++c) {
      double s = 0.0;
      for (int64_t i : kv.second) s += (double)grads[i * D + c];
      const float g = (float)s;
      const float p = lr * g;
      w[c] = w[c] - p;
    }
  }
  put_done(t, rows);
  return kOk;
}

// rows_out[i] = row of keys[i], or -1 if absent. Never inserts.
int oracle_lookup_rows(oracle_table* h, const uint64_t* keys, int64_t n, int64_t* rows_out) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (n < 0 || (n > 0 && (keys == nullptr || rows_out == nullptr))) return kEinval;
  for (int64_t i = 0; i < n; ++i) {
    uint32_t r;
    rows_out[i] = find_row(t, keys[i], &r) ? (int64_t)r : -1;
  }
  return kOk;
}

// Copies rows[j] (each in [0, size)) into out[j*dim ...] and its accumulator
// into state_out[j] (either output may be NULL).
int oracle_read_rows(oracle_table* h, const int64_t* rows, int64_t nr, float* out, float* state_out) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (nr < 0 || (nr > 0 && rows == nullptr)) return kEinval;
  for (int64_t j = 0; j < nr; ++j)
    if (rows[j] < 0 || rows[j] >= t.size) return kEinval;
  for (int64_t j = 0; j < nr; ++j) {
    const uint32_t r = (uint32_t)rows[j];
    if (out)
      for (int32_t c = 0; c < t.dim; ++c) out[j * t.dim + c] = read_elem(t, r, c);
    if (state_out) {
      auto it = t.accum.find(r);
      state_out[j] = it == t.accum.end() ? 0.0f : it->second;
    }
  }
  return kOk;
}

// count_out[j] = staleness count c_k (R8) of row rows[j]; 0 when not tracked.
int oracle_staleness(oracle_table* h, const int64_t* rows, int64_t nr, uint32_t* count_out) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (nr < 0 || (nr > 0 && (rows == nullptr || count_out == nullptr))) return kEinval;
  for (int64_t j = 0; j < nr; ++j) {
    if (rows[j] < 0 || rows[j] >= t.size) return kEinval;
    auto it = t.stale.find((uint32_t)rows[j]);
    count_out[j] = it == t.stale.end() ? 0u : it->second;
  }
  return kOk;
}

// key_out[j] = key stored in row rows[j].
int oracle_row_keys(oracle_table* h, const int64_t* rows, int64_t nr, uint64_t* key_out) {
  Table& t = *reinterpret_cast<Table*>(h);
  if (nr < 0 || (nr > 0 && (rows == nullptr || key_out == nullptr))) return kEinval;
  for (int64_t j = 0; j < nr; ++j) {
    if (rows[j] < 0 || rows[j] >= t.size) return kEinval;
    key_out[j] = t.row_key[(size_t)rows[j]];
  }
  return kOk;
}

}  // extern "C"

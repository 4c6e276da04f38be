// Cache maintainer under the LCBFU policy (Sec. 5.4): host data structures
// that decide which cached intermediate states to evict, where new states
// go, and which vector-DB rows to drop.  The device-side effects (state pool
// table, row compaction, new rows) are applied by the pool kernels and
// nv_cache_insert from the plan this code returns.
//
// Every cached state i has the score f_i * K_i: f_i counts the requests
// served from it (starting at 1 for the generation that stored it) and K_i
// is the number of denoising steps it was saved after.  A min-heap over
// (score, insertion sequence) yields the next victim in O(log n); a served
// request raises f_i and moves the state down the heap.
#include <algorithm>
#include <cstdint>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "../../include/nv.h"

namespace nv {
void set_error(const std::string& msg);
void clear_error();
}  // namespace nv

#define LC_CHECK(cond, msg)        \
  do {                             \
    if (!(cond)) {                 \
      ::nv::set_error(msg);        \
      return NV_ERR_INVALID_ARG;   \
    }                              \
  } while (0)

typedef std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> MinQueue;

struct nv_lcbfu {
  int S = 0;
  int32_t slot_k[16] = {};
  int64_t cap = 0, ecap = 0;
  // per pool state (indexed by its pool slot)
  std::vector<int32_t> st_entry;
  std::vector<int32_t> st_slot;
  std::vector<int64_t> st_f, st_seq, st_pos;  // st_pos: heap position, -1 = free
  std::vector<int32_t> heap;                  // pool slots, min on (f * K, seq)
  // per entry (prompt)
  std::vector<int32_t> table;                 // [ecap][S] pool slot or -1
  std::vector<int32_t> entry_row;             // row in the vector DB or -1
  std::vector<int32_t> entry_live;            // states still stored
  std::vector<int32_t> rows;                  // vector-DB row -> entry
  MinQueue free_pool, free_entries;
  int64_t seq = 0, evicted = 0, dropped = 0;

  int64_t key(int32_t p) const { return st_f[p] * slot_k[st_slot[p]]; }
  bool less(int32_t a, int32_t b) const {
    const int64_t ka = key(a), kb = key(b);
    return ka != kb ? ka < kb : st_seq[a] < st_seq[b];
  }
  void place(int64_t i, int32_t p) {
    heap[i] = p;
    st_pos[p] = i;
  }
  void sift_up(int64_t i) {
    const int32_t p = heap[i];
    while (i > 0) {
      const int64_t up = (i - 1) / 2;
      if (!less(p, heap[up])) break;
      place(i, heap[up]);
      i = up;
    }
    place(i, p);
  }
  void sift_down(int64_t i) {
    const int32_t p = heap[i];
    const int64_t n = (int64_t)heap.size();
    for (;;) {
      int64_t c = 2 * i + 1;
      if (c >= n) break;
      if (c + 1 < n && less(heap[c + 1], heap[c])) ++c;
      if (!less(heap[c], p)) break;
      place(i, heap[c]);
      i = c;
    }
    place(i, p);
  }
  int32_t pop_min() {
    const int32_t p = heap[0];
    const int32_t last = heap.back();
    heap.pop_back();
    if (!heap.empty()) {
      heap[0] = last;
      st_pos[last] = 0;
      sift_down(0);
    }
    st_pos[p] = -1;
    return p;
  }
  void push(int32_t p) {
    heap.push_back(p);
    sift_up((int64_t)heap.size() - 1);
  }
};

extern "C" int32_t nv_lcbfu_create(int32_t n_slots, const int32_t* slot_k, int64_t state_capacity,
                                   int64_t entry_capacity, nv_lcbfu** out) {
  nv::clear_error();
  LC_CHECK(out, "null out");
  *out = nullptr;
  LC_CHECK(n_slots >= 1 && n_slots <= 16 && slot_k, "need 1..16 slots");
  for (int s = 0; s < n_slots; ++s) {
    LC_CHECK(slot_k[s] >= 1, "slot_k must be >= 1");
    for (int t = 0; t < s; ++t) LC_CHECK(slot_k[s] != slot_k[t], "slot_k values must differ");
  }
  LC_CHECK(state_capacity >= 1 && state_capacity < (int64_t(1) << 31),
           "state_capacity must be in [1, 2^31)");
  LC_CHECK(entry_capacity >= state_capacity && entry_capacity < (int64_t(1) << 31),
           "entry_capacity must be in [state_capacity, 2^31)");
  nv_lcbfu* h = new (std::nothrow) nv_lcbfu();
  if (!h) {
    nv::set_error("host allocation failed");
    return NV_ERR_OUT_OF_MEMORY;
  }
  try {
    h->S = n_slots;
    for (int s = 0; s < n_slots; ++s) h->slot_k[s] = slot_k[s];
    h->cap = state_capacity;
    h->ecap = entry_capacity;
    h->st_entry.assign(state_capacity, -1);
    h->st_slot.assign(state_capacity, 0);
    h->st_f.assign(state_capacity, 0);
    h->st_seq.assign(state_capacity, 0);
    h->st_pos.assign(state_capacity, -1);
    h->heap.reserve(state_capacity);
    h->table.assign((size_t)entry_capacity * n_slots, -1);
    h->entry_row.assign(entry_capacity, -1);
    h->entry_live.assign(entry_capacity, 0);
    h->rows.reserve(entry_capacity);
    std::vector<int64_t> ids(state_capacity);
    for (int64_t i = 0; i < state_capacity; ++i) ids[i] = i;
    h->free_pool = MinQueue(std::greater<int64_t>(), std::move(ids));
    std::vector<int64_t> eids(entry_capacity);
    for (int64_t i = 0; i < entry_capacity; ++i) eids[i] = i;
    h->free_entries = MinQueue(std::greater<int64_t>(), std::move(eids));
  } catch (const std::bad_alloc&) {
    delete h;
    nv::set_error("host allocation failed");
    return NV_ERR_OUT_OF_MEMORY;
  }
  *out = h;
  return NV_OK;
}

extern "C" void nv_lcbfu_destroy(nv_lcbfu* h) { delete h; }

extern "C" int32_t nv_lcbfu_access(nv_lcbfu* h, int32_t B, const int64_t* row, const int32_t* k) {
  nv::clear_error();
  LC_CHECK(h && row && k && B >= 0, "null handle / arrays or negative B");
  std::vector<int32_t> hit(B, -1);
  for (int b = 0; b < B; ++b) {
    if (k[b] <= 0) continue;
    LC_CHECK(row[b] >= 0 && row[b] < (int64_t)h->rows.size(), "row out of range");
    int s = -1;
    for (int t = 0; t < h->S; ++t)
      if (h->slot_k[t] == k[b]) s = t;
    LC_CHECK(s >= 0, "k is not a slot's K");
    const int32_t p = h->table[(size_t)h->rows[row[b]] * h->S + s];
    LC_CHECK(p >= 0, "k names a hole of that row's prompt");
    hit[b] = p;
  }
  for (int b = 0; b < B; ++b)
    if (hit[b] >= 0) {
      ++h->st_f[hit[b]];
      h->sift_down(h->st_pos[hit[b]]);
    }
  return NV_OK;
}

extern "C" int32_t nv_lcbfu_insert(nv_lcbfu* h, int32_t m, int32_t* entry_out, int32_t* state_out,
                                   int64_t* move_src, int64_t* move_dst, int32_t* n_moves,
                                   int32_t* upd, int32_t* n_upd, int64_t* n_kept) {
  nv::clear_error();
  LC_CHECK(h && entry_out && state_out && move_src && move_dst && n_moves && upd && n_upd &&
               n_kept, "null handle or output");
  LC_CHECK(m >= 1 && (int64_t)m * h->S <= h->cap, "m * n_slots must be in [1, state_capacity]");
  const int S = h->S;
  const int64_t need = (int64_t)h->heap.size() + (int64_t)m * S - h->cap;
  std::vector<int32_t> touched, dead;
  for (int64_t v = 0; v < need; ++v) {
    const int32_t p = h->pop_min();
    const int32_t e = h->st_entry[p];
    h->table[(size_t)e * S + h->st_slot[p]] = -1;
    h->st_entry[p] = -1;
    h->free_pool.push(p);
    ++h->evicted;
    touched.push_back(e);
    if (--h->entry_live[e] == 0) dead.push_back(e);
  }
  // drop prompts with no state left; live rows from the end fill their rows
  const int64_t n_rows = (int64_t)h->rows.size();
  const int64_t kept = n_rows - (int64_t)dead.size();
  std::vector<int64_t> holes;
  for (int32_t e : dead)
    if (h->entry_row[e] < kept) holes.push_back(h->entry_row[e]);
  std::sort(holes.begin(), holes.end());
  int32_t nm = 0;
  for (int64_t r = kept; r < n_rows; ++r) {
    const int32_t e = h->rows[r];
    if (h->entry_live[e] == 0) continue;
    const int64_t to = holes[nm];
    move_src[nm] = r;
    move_dst[nm] = to;
    ++nm;
    h->rows[to] = e;
    h->entry_row[e] = (int32_t)to;
  }
  h->rows.resize(kept);
  for (int32_t e : dead) {
    h->entry_row[e] = -1;
    h->free_entries.push(e);
  }
  h->dropped += (int64_t)dead.size();
  // store the new prompts: lowest free ids and pool slots first
  for (int i = 0; i < m; ++i) {
    const int32_t e = (int32_t)h->free_entries.top();
    h->free_entries.pop();
    for (int s = 0; s < S; ++s) {
      const int32_t p = (int32_t)h->free_pool.top();
      h->free_pool.pop();
      h->st_entry[p] = e;
      h->st_slot[p] = s;
      h->st_f[p] = 1;
      h->st_seq[p] = h->seq++;
      h->push(p);
      h->table[(size_t)e * S + s] = p;
      state_out[(size_t)i * S + s] = p;
    }
    h->entry_live[e] = S;
    h->entry_row[e] = (int32_t)h->rows.size();
    h->rows.push_back(e);
    entry_out[i] = e;
    touched.push_back(e);
  }
  std::sort(touched.begin(), touched.end());
  touched.erase(std::unique(touched.begin(), touched.end()), touched.end());
  for (size_t u = 0; u < touched.size(); ++u) {
    int32_t* rec = upd + u * (size_t)(1 + S);
    rec[0] = touched[u];
    for (int s = 0; s < S; ++s) rec[1 + s] = h->table[(size_t)touched[u] * S + s];
  }
  *n_moves = nm;
  *n_upd = (int32_t)touched.size();
  *n_kept = kept;
  return NV_OK;
}

extern "C" int32_t nv_lcbfu_info(const nv_lcbfu* h, int64_t* info) {
  nv::clear_error();
  LC_CHECK(h && info, "null handle or info");
  info[0] = (int64_t)h->rows.size();
  info[1] = (int64_t)h->heap.size();
  info[2] = h->evicted;
  info[3] = h->dropped;
  info[4] = h->seq;
  return NV_OK;
}

extern "C" int32_t nv_lcbfu_export(const nv_lcbfu* h, int32_t* table, int32_t* rows,
                                   int64_t* counts) {
  nv::clear_error();
  LC_CHECK(h, "null handle");
  if (table) std::copy(h->table.begin(), h->table.end(), table);
  if (rows) std::copy(h->rows.begin(), h->rows.end(), rows);
  if (counts)
    for (int64_t p = 0; p < h->cap; ++p) counts[p] = h->st_pos[p] >= 0 ? h->st_f[p] : 0;
  return NV_OK;
}

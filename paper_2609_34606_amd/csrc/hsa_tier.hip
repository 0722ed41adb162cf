// Host-managed tier of the KV cache (Sec. 3.2 "Cache hierarchy and
// dataflow"): L1 is the device pool's slots, L2 pinned host memory. Pages
// that the retrieval does not select move to L2 when L1 is full (least
// recently used first) and come back before the attention that needs them.
//
// The manager owns the placement of logical pages. It keeps, per batch entry
// and logical page, where the page lives (an L1 slot or an L2 slot), a
// last-use tick, and mirrors the L1 slots of the device page table. All copies
// (one contiguous block per page for keys and one for values: a slot holds
// every head of a page) and the page-table updates go on the caller's stream
// in order, so kernels launched after a call on that stream see the pages in
// place. Without device pointers ("plan-only") the same bookkeeping runs and
// no copy is issued, which lets the policy be checked without a GPU.
#include <stdint.h>
#include <string.h>

#include <vector>

#include "hsa_kernels.h"

struct hsa_tier {
  int32_t batch, max_pages, l1_slots, l2_slots;
  int32_t n_placed = 0;
  size_t k_bytes, v_bytes;   // bytes of one slot of the key / value pool
  char* dev_k;               // device pool (NULL: plan-only)
  char* dev_v;
  int32_t* dev_table;        // device page table [batch, max_pages]
  char* host_k;              // pinned host slots
  char* host_v;
  // per (b, page): -1 absent, >= 0 an L1 slot, <= -2 the L2 slot -(loc + 2)
  std::vector<int32_t> loc;
  std::vector<uint64_t> tick;
  std::vector<int32_t> l1_owner;   // per L1 slot: b * max_pages + page, or -1
  std::vector<int32_t> l2_owner;   // per L2 slot
  std::vector<int32_t> table;      // host mirror of the device page table
  uint64_t now = 0;
  int64_t n_evict = 0, n_fetch = 0;
};

namespace {

hsa_status_t copy(void* dst, const void* src, size_t n, hipMemcpyKind kind, hipStream_t s) {
  return hipMemcpyAsync(dst, src, n, kind, s) == hipSuccess ? HSA_OK : HSA_ERR_DEVICE;
}

bool live(const hsa_tier* t) { return t->dev_k != nullptr; }

// One page-table entry, passed by value (a copy from host memory that later
// calls change could run after the change).
__global__ void set_entry_kernel(int32_t* dst, int32_t value) { *dst = value; }

// Publishes the L1 slot of page index g in the device page table.
hsa_status_t publish(hsa_tier* t, int g, hipStream_t s) {
  if (!live(t)) return HSA_OK;
  set_entry_kernel<<<1, 1, 0, s>>>(t->dev_table + g, t->table[g]);
  return hipGetLastError() == hipSuccess ? HSA_OK : HSA_ERR_DEVICE;
}

// A free L1 slot, moving the least recently used unpinned resident page to a
// free L2 slot first when none is free. pinned: page indices that must stay.
hsa_status_t free_l1(hsa_tier* t, const std::vector<char>& pinned, int* slot, hipStream_t s) {
  for (int i = 0; i < t->l1_slots; ++i)
    if (t->l1_owner[i] < 0) {
      *slot = i;
      return HSA_OK;
    }
  int victim = -1;
  for (int i = 0; i < t->l1_slots; ++i) {
    const int g = t->l1_owner[i];
    if (pinned[g]) continue;
    if (victim < 0 || t->tick[g] < t->tick[t->l1_owner[victim]]) victim = i;
  }
  if (victim < 0) return HSA_ERR_UNSUPPORTED;  // every L1 page is needed at once
  int l2 = -1;
  for (int i = 0; i < t->l2_slots; ++i)
    if (t->l2_owner[i] < 0) {
      l2 = i;
      break;
    }
  if (l2 < 0) return HSA_ERR_UNSUPPORTED;      // L2 is full
  const int g = t->l1_owner[victim];
  if (live(t)) {
    hsa_status_t st = copy(t->host_k + (size_t)l2 * t->k_bytes, t->dev_k + (size_t)victim * t->k_bytes,
                           t->k_bytes, hipMemcpyDeviceToHost, s);
    if (st == HSA_OK)
      st = copy(t->host_v + (size_t)l2 * t->v_bytes, t->dev_v + (size_t)victim * t->v_bytes, t->v_bytes,
                hipMemcpyDeviceToHost, s);
    if (st != HSA_OK) return st;
  }
  t->l2_owner[l2] = g;
  t->l1_owner[victim] = -1;
  t->loc[g] = -(l2 + 2);
  ++t->n_evict;
  *slot = victim;
  return HSA_OK;
}

}  // namespace

extern "C" {

hsa_status_t hsa_tier_create(const hsa_config_t* cfg, const hsa_kv_pool_t* pool, void* host_k,
                             void* host_v, int32_t l2_slots, hsa_tier_t** out) {
  if (!cfg || !pool || !out) return HSA_ERR_INVALID_ARG;
  if (cfg->batch < 1 || cfg->num_heads < 1 || cfg->head_dim < 1 || cfg->page_size < 1)
    return HSA_ERR_INVALID_ARG;
  if (pool->num_slots < 1 || pool->max_pages < 1 || l2_slots < 0) return HSA_ERR_INVALID_ARG;
  const bool plan_only = pool->k == nullptr;
  if (!plan_only && (!pool->v || !pool->page_table || (l2_slots > 0 && (!host_k || !host_v))))
    return HSA_ERR_INVALID_ARG;
  hsa_tier* t = new hsa_tier();
  t->batch = cfg->batch;
  t->max_pages = pool->max_pages;
  t->l1_slots = pool->num_slots;
  t->l2_slots = l2_slots;
  const size_t esize = cfg->dtype == HSA_DTYPE_BF16 ? 2 : 4;
  t->k_bytes = t->v_bytes = (size_t)cfg->num_heads * cfg->page_size * cfg->head_dim * esize;
  t->dev_k = static_cast<char*>(const_cast<void*>(pool->k));
  t->dev_v = static_cast<char*>(const_cast<void*>(pool->v));
  t->dev_table = const_cast<int32_t*>(pool->page_table);
  t->host_k = static_cast<char*>(host_k);
  t->host_v = static_cast<char*>(host_v);
  const size_t n = (size_t)cfg->batch * pool->max_pages;
  t->loc.assign(n, -1);
  t->tick.assign(n, 0);
  t->table.assign(n, -1);
  t->l1_owner.assign(pool->num_slots, -1);
  t->l2_owner.assign(l2_slots, -1);
  *out = t;
  return HSA_OK;
}

void hsa_tier_destroy(hsa_tier_t* t) { delete t; }

hsa_status_t hsa_tier_place(hsa_tier_t* t, int32_t b, int32_t page, int32_t* slot, void* stream) {
  if (!t || !slot) return HSA_ERR_INVALID_ARG;
  if (b < 0 || b >= t->batch || page < 0 || page >= t->max_pages) return HSA_ERR_OUT_OF_RANGE;
  const int g = b * t->max_pages + page;
  if (t->loc[g] != -1) return HSA_ERR_INVALID_ARG;  // already placed
  // one host slot always stays free, so that a fetch can move a page out
  // before the page it brings back leaves its host slot
  const int cap = t->l2_slots > 0 ? t->l1_slots + t->l2_slots - 1 : t->l1_slots;
  if (t->n_placed >= cap) return HSA_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<char> pinned(t->loc.size(), 0);
  int sl = -1;
  hsa_status_t st = free_l1(t, pinned, &sl, s);
  if (st != HSA_OK) return st;
  t->l1_owner[sl] = g;
  t->loc[g] = sl;
  ++t->n_placed;
  t->tick[g] = ++t->now;
  t->table[g] = sl;
  *slot = sl;
  return publish(t, g, s);
}

hsa_status_t hsa_tier_fetch(hsa_tier_t* t, const int32_t* pages, int32_t n_per_batch, void* stream) {
  if (!t || (n_per_batch > 0 && !pages) || n_per_batch < 0) return HSA_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // every listed page is pinned for this call and becomes the most recent
  std::vector<char> pinned(t->loc.size(), 0);
  for (int b = 0; b < t->batch; ++b)
    for (int i = 0; i < n_per_batch; ++i) {
      const int p = pages[(size_t)b * n_per_batch + i];
      if (p < 0) continue;
      if (p >= t->max_pages) return HSA_ERR_OUT_OF_RANGE;
      const int g = b * t->max_pages + p;
      if (t->loc[g] == -1) return HSA_ERR_INVALID_ARG;  // never placed
      pinned[g] = 1;
    }
  const uint64_t use = ++t->now;
  for (size_t g = 0; g < pinned.size(); ++g) {
    if (!pinned[g]) continue;
    t->tick[g] = use;
    if (t->loc[g] >= 0) continue;
    const int l2 = -(t->loc[g] + 2);
    int sl = -1;
    hsa_status_t st = free_l1(t, pinned, &sl, s);
    if (st != HSA_OK) return st;
    if (live(t)) {
      st = copy(t->dev_k + (size_t)sl * t->k_bytes, t->host_k + (size_t)l2 * t->k_bytes, t->k_bytes,
                hipMemcpyHostToDevice, s);
      if (st == HSA_OK)
        st = copy(t->dev_v + (size_t)sl * t->v_bytes, t->host_v + (size_t)l2 * t->v_bytes, t->v_bytes,
                  hipMemcpyHostToDevice, s);
      if (st != HSA_OK) return st;
    }
    t->l2_owner[l2] = -1;
    t->l1_owner[sl] = (int32_t)g;
    t->loc[g] = sl;
    t->table[g] = sl;
    ++t->n_fetch;
    if ((st = publish(t, (int)g, s)) != HSA_OK) return st;
  }
  return HSA_OK;
}

int32_t hsa_tier_locate(const hsa_tier_t* t, int32_t b, int32_t page) {
  if (!t || b < 0 || b >= t->batch || page < 0 || page >= t->max_pages) return -1;
  return t->loc[(size_t)b * t->max_pages + page];
}

void hsa_tier_counters(const hsa_tier_t* t, int64_t* evictions, int64_t* fetches) {
  if (!t) return;
  if (evictions) *evictions = t->n_evict;
  if (fetches) *fetches = t->n_fetch;
}

}  // extern "C"

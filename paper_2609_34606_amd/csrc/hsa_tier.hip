// Host-managed tiers of the KV cache (Sec. 3.2 "Cache hierarchy and
// dataflow"): L1 is the device pool's slots, L2 pinned host memory, L3 a file
// (an NVMe drive). Pages leave L1 least recently used first when a slot is
// needed, L2 spills to L3 the same way, and the pages a forward pass needs
// come back to L1 before the kernels that read them.
//
// The manager owns the placement of logical pages. It keeps, per batch entry
// and logical page, where the page lives, a last-use tick, the owner of every
// slot, and a mirror of the device page table. A slot holds every head of a
// page (one contiguous key block and one value block).
//
// Streams. The caller's compute stream carries place, fetch and the kernels
// that read the pool; host-to-device copies of a fetch and the page-table
// updates go on it. Device-to-host copies (pages leaving L1) go on an
// internal stream, so that a page going out and one coming in use both
// directions of the link at once. A prefetch runs on a side stream of the
// caller's: its copies overlap the kernels of the compute stream, it never
// moves a page the kernels may read (those of the last fetch and pages placed
// since), it starts after the compute stream has passed the last fetch, and
// the next fetch waits for it. Every async copy records an event on the slot
// it touches (pool slot, host slot, staging buffer); the next copy or host
// access of that slot waits for it, so copies issued on different streams
// never overlap on one slot. Without device pointers ("plan-only") the same
// bookkeeping runs and no copy, event or file access is issued.
#include <errno.h>
#include <fcntl.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <string>
#include <vector>

#include "hsa_kernels.h"

namespace {

// One event per slot, recorded after the last async copy that touched it.
struct SlotEvents {
  std::vector<hipEvent_t> ev;
  std::vector<char> set;
};

}  // namespace

struct hsa_tier {
  int32_t batch, max_pages, l1_slots, l2_slots, l3_slots;
  int32_t n_placed = 0;
  size_t k_bytes, v_bytes;   // bytes of one slot of the key / value pool
  char* dev_k;               // device pool (NULL: plan-only)
  char* dev_v;
  int32_t* dev_table;        // device page table [batch, max_pages]
  char* host_k;              // pinned host slots (L2)
  char* host_v;
  int fd = -1;               // L3 file: slot i at offset i * (k_bytes + v_bytes)
  char* bounce[2] = {nullptr, nullptr};   // pinned staging of L3 reads
  int next_bounce = 0;
  // per (b, page): -1 absent, >= 0 an L1 slot, -(2 + i) L2 slot i,
  // -(2 + l2_slots + i) L3 slot i
  std::vector<int32_t> loc;
  std::vector<uint64_t> tick;
  std::vector<char> held;          // pages the compute stream's kernels may read
  std::vector<int32_t> l1_owner;   // per slot: b * max_pages + page, or -1
  std::vector<int32_t> l2_owner;
  std::vector<int32_t> l3_owner;
  std::vector<int32_t> table;      // host mirror of the device page table
  uint64_t now = 0;
  hsa_tier_stats_t stats{};
  // live mode only
  hipStream_t out_stream = nullptr;        // device-to-host copies
  SlotEvents l1_ev, l2_ev, bounce_ev;
  hipEvent_t ev_start = nullptr, ev_out_done = nullptr, ev_fetch = nullptr,
             ev_prefetch = nullptr;
  bool fetch_recorded = false, prefetch_pending = false;
};

namespace {

bool live(const hsa_tier* t) { return t->dev_k != nullptr; }

int l2_code(int i) { return -(2 + i); }
int l3_code(const hsa_tier* t, int i) { return -(2 + t->l2_slots + i); }
int l2_index(const hsa_tier* t, int loc) {
  const int i = -(loc + 2);
  return (loc <= -2 && i < t->l2_slots) ? i : -1;
}
int l3_index(const hsa_tier* t, int loc) {
  const int i = -(loc + 2) - t->l2_slots;
  return (loc <= -2 && i >= 0) ? i : -1;
}

bool ok(hipError_t e) { return e == hipSuccess; }

hsa_status_t make_events(SlotEvents& e, int n) {
  e.ev.assign(n, nullptr);
  e.set.assign(n, 0);
  for (int i = 0; i < n; ++i)
    if (!ok(hipEventCreateWithFlags(&e.ev[i], hipEventDisableTiming))) return HSA_ERR_DEVICE;
  return HSA_OK;
}

void drop_events(SlotEvents& e) {
  for (size_t i = 0; i < e.ev.size(); ++i)
    if (e.ev[i]) {
      if (e.set[i]) hipEventSynchronize(e.ev[i]);
      hipEventDestroy(e.ev[i]);
    }
  e.ev.clear();
  e.set.clear();
}

// Stream s waits for the last copy on slot i.
hsa_status_t after(hipStream_t s, SlotEvents& e, int i) {
  if (!e.set[i]) return HSA_OK;
  return ok(hipStreamWaitEvent(s, e.ev[i], 0)) ? HSA_OK : HSA_ERR_DEVICE;
}

// Records the copy just issued on s as the last one on slot i.
hsa_status_t mark(hipStream_t s, SlotEvents& e, int i) {
  e.set[i] = 1;
  return ok(hipEventRecord(e.ev[i], s)) ? HSA_OK : HSA_ERR_DEVICE;
}

// The host waits for the last copy on slot i (before reading or writing it).
hsa_status_t host_wait(SlotEvents& e, int i) {
  if (!e.set[i]) return HSA_OK;
  return ok(hipEventSynchronize(e.ev[i])) ? HSA_OK : HSA_ERR_DEVICE;
}

hsa_status_t copy(void* dst, const void* src, size_t n, hipMemcpyKind kind, hipStream_t s) {
  return ok(hipMemcpyAsync(dst, src, n, kind, s)) ? HSA_OK : HSA_ERR_DEVICE;
}

hsa_status_t file_io(int fd, char* buf, size_t n, off_t off, bool write) {
  while (n > 0) {
    const ssize_t r = write ? pwrite(fd, buf, n, off) : pread(fd, buf, n, off);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return HSA_ERR_IO;
    buf += r;
    off += r;
    n -= (size_t)r;
  }
  return HSA_OK;
}

off_t l3_offset(const hsa_tier* t, int i) { return (off_t)i * (off_t)(t->k_bytes + t->v_bytes); }

// One page-table entry, passed by value (a copy from host memory that later
// calls change could run after the change).
__global__ void set_entry_kernel(int32_t* dst, int32_t value) { *dst = value; }

// Publishes the L1 slot of page index g in the device page table.
hsa_status_t publish(hsa_tier* t, int g, hipStream_t s) {
  if (!live(t)) return HSA_OK;
  set_entry_kernel<<<1, 1, 0, s>>>(t->dev_table + g, t->table[g]);
  return ok(hipGetLastError()) ? HSA_OK : HSA_ERR_DEVICE;
}

// A free L3 slot, or -1.
int free_l3(const hsa_tier* t) {
  for (int i = 0; i < t->l3_slots; ++i)
    if (t->l3_owner[i] < 0) return i;
  return -1;
}

// A free L2 slot; when none is free, the least recently used L2 page that is
// not pinned is written to a free L3 slot first (the host waits for the copy
// that filled its host slot).
hsa_status_t take_l2(hsa_tier* t, const std::vector<char>& pinned, int* out) {
  for (int i = 0; i < t->l2_slots; ++i)
    if (t->l2_owner[i] < 0) {
      *out = i;
      return HSA_OK;
    }
  const int c = free_l3(t);
  if (c < 0) return HSA_ERR_UNSUPPORTED;   // every tier is full
  int w = -1;
  for (int i = 0; i < t->l2_slots; ++i) {
    const int g = t->l2_owner[i];
    if (pinned[g]) continue;
    if (w < 0 || t->tick[g] < t->tick[t->l2_owner[w]]) w = i;
  }
  if (w < 0) return HSA_ERR_UNSUPPORTED;   // every L2 page is needed now
  if (live(t)) {
    hsa_status_t st = host_wait(t->l2_ev, w);
    if (st == HSA_OK)
      st = file_io(t->fd, t->host_k + (size_t)w * t->k_bytes, t->k_bytes, l3_offset(t, c), true);
    if (st == HSA_OK)
      st = file_io(t->fd, t->host_v + (size_t)w * t->v_bytes, t->v_bytes,
                   l3_offset(t, c) + (off_t)t->k_bytes, true);
    if (st != HSA_OK) return st;
  }
  const int g = t->l2_owner[w];
  t->l3_owner[c] = g;
  t->l2_owner[w] = -1;
  t->loc[g] = l3_code(t, c);
  ++t->stats.spills;
  *out = w;
  return HSA_OK;
}

// Moves the page in L1 slot v straight to L3 slot c through a staging page
// (when every L2 page is needed by the current call).
hsa_status_t l1_to_l3(hsa_tier* t, int v, int c) {
  if (!live(t)) return HSA_OK;
  const int j = t->next_bounce;
  t->next_bounce ^= 1;
  hipStream_t e = t->out_stream;
  hsa_status_t st = host_wait(t->bounce_ev, j);
  if (st == HSA_OK) st = after(e, t->l1_ev, v);
  if (st == HSA_OK)
    st = copy(t->bounce[j], t->dev_k + (size_t)v * t->k_bytes, t->k_bytes, hipMemcpyDeviceToHost, e);
  if (st == HSA_OK)
    st = copy(t->bounce[j] + t->k_bytes, t->dev_v + (size_t)v * t->v_bytes, t->v_bytes,
              hipMemcpyDeviceToHost, e);
  if (st == HSA_OK) st = mark(e, t->l1_ev, v);
  if (st == HSA_OK) st = mark(e, t->bounce_ev, j);
  if (st == HSA_OK) st = host_wait(t->bounce_ev, j);
  if (st == HSA_OK) st = file_io(t->fd, t->bounce[j], t->k_bytes + t->v_bytes, l3_offset(t, c), true);
  return st;
}

// A free L1 slot, moving the least recently used unpinned resident page down
// a tier first when none is free: to L2 (device-to-host copy on the internal
// stream), or to L3 when no L2 page may make room. Fails before changing
// anything when no page may move.
hsa_status_t take_l1(hsa_tier* t, const std::vector<char>& pinned, int* out) {
  for (int i = 0; i < t->l1_slots; ++i)
    if (t->l1_owner[i] < 0) {
      *out = i;
      return HSA_OK;
    }
  int v = -1;
  for (int i = 0; i < t->l1_slots; ++i) {
    const int g = t->l1_owner[i];
    if (pinned[g]) continue;
    if (v < 0 || t->tick[g] < t->tick[t->l1_owner[v]]) v = i;
  }
  if (v < 0) return HSA_ERR_UNSUPPORTED;   // every L1 page is needed at once
  const int g = t->l1_owner[v];
  int a = -1;
  hsa_status_t st = take_l2(t, pinned, &a);
  if (st == HSA_ERR_UNSUPPORTED) {
    const int c = free_l3(t);
    if (c < 0) return st;
    if ((st = l1_to_l3(t, v, c)) != HSA_OK) return st;
    t->l3_owner[c] = g;
    t->l1_owner[v] = -1;
    t->loc[g] = l3_code(t, c);
    ++t->stats.evictions;
    ++t->stats.spills;
    *out = v;
    return HSA_OK;
  }
  if (st != HSA_OK) return st;
  if (live(t)) {
    hipStream_t e = t->out_stream;
    st = after(e, t->l1_ev, v);
    if (st == HSA_OK) st = after(e, t->l2_ev, a);
    if (st == HSA_OK)
      st = copy(t->host_k + (size_t)a * t->k_bytes, t->dev_k + (size_t)v * t->k_bytes, t->k_bytes,
                hipMemcpyDeviceToHost, e);
    if (st == HSA_OK)
      st = copy(t->host_v + (size_t)a * t->v_bytes, t->dev_v + (size_t)v * t->v_bytes, t->v_bytes,
                hipMemcpyDeviceToHost, e);
    if (st == HSA_OK) st = mark(e, t->l1_ev, v);
    if (st == HSA_OK) st = mark(e, t->l2_ev, a);
    if (st != HSA_OK) return st;
  }
  t->l2_owner[a] = g;
  t->l1_owner[v] = -1;
  t->loc[g] = l2_code(a);
  ++t->stats.evictions;
  *out = v;
  return HSA_OK;
}

// Brings page index g into L1 (host-to-device copy on s).
hsa_status_t bring(hsa_tier* t, int g, const std::vector<char>& pinned, hipStream_t s) {
  const int loc = t->loc[g];
  if (loc >= 0) return HSA_OK;
  const int i2 = l2_index(t, loc), i3 = l3_index(t, loc);
  int sl = -1, j = -1;
  hsa_status_t st;
  if (i3 >= 0) {
    // read into a staging buffer first: the L3 slot is then free for a spill
    // that making room in L1 may cause
    j = t->next_bounce;
    t->next_bounce ^= 1;
    if (live(t)) {
      st = host_wait(t->bounce_ev, j);
      if (st == HSA_OK) st = file_io(t->fd, t->bounce[j], t->k_bytes, l3_offset(t, i3), false);
      if (st == HSA_OK)
        st = file_io(t->fd, t->bounce[j] + t->k_bytes, t->v_bytes, l3_offset(t, i3) + (off_t)t->k_bytes,
                     false);
      if (st != HSA_OK) return st;
    }
    t->l3_owner[i3] = -1;
    st = take_l1(t, pinned, &sl);
    if (st != HSA_OK) {
      t->l3_owner[i3] = g;   // nothing was written over it
      return st;
    }
    ++t->stats.reloads;
  } else {
    st = take_l1(t, pinned, &sl);
    if (st != HSA_OK) return st;
  }
  if (live(t)) {
    const char* sk = i3 >= 0 ? t->bounce[j] : t->host_k + (size_t)i2 * t->k_bytes;
    const char* sv = i3 >= 0 ? t->bounce[j] + t->k_bytes : t->host_v + (size_t)i2 * t->v_bytes;
    st = after(s, t->l1_ev, sl);
    if (st == HSA_OK && i2 >= 0) st = after(s, t->l2_ev, i2);
    if (st == HSA_OK)
      st = copy(t->dev_k + (size_t)sl * t->k_bytes, sk, t->k_bytes, hipMemcpyHostToDevice, s);
    if (st == HSA_OK)
      st = copy(t->dev_v + (size_t)sl * t->v_bytes, sv, t->v_bytes, hipMemcpyHostToDevice, s);
    if (st == HSA_OK) st = mark(s, t->l1_ev, sl);
    if (st == HSA_OK) st = i3 >= 0 ? mark(s, t->bounce_ev, j) : mark(s, t->l2_ev, i2);
    if (st != HSA_OK) return st;
  }
  if (i2 >= 0) t->l2_owner[i2] = -1;
  t->l1_owner[sl] = g;
  t->loc[g] = sl;
  t->table[g] = sl;
  ++t->stats.fetches;
  return publish(t, g, s);
}

// Orders a call's copies after the work already on s (and after `wait`, if
// given): the internal stream starts where s is now.
hsa_status_t begin(hsa_tier* t, hipStream_t s, hipEvent_t wait) {
  if (!live(t)) return HSA_OK;
  if (wait && !ok(hipStreamWaitEvent(s, wait, 0))) return HSA_ERR_DEVICE;
  if (!ok(hipEventRecord(t->ev_start, s))) return HSA_ERR_DEVICE;
  return ok(hipStreamWaitEvent(t->out_stream, t->ev_start, 0)) ? HSA_OK : HSA_ERR_DEVICE;
}

// Work issued on s after the call starts after all of the call's copies.
hsa_status_t end(hsa_tier* t, hipStream_t s) {
  if (!live(t)) return HSA_OK;
  if (!ok(hipEventRecord(t->ev_out_done, t->out_stream))) return HSA_ERR_DEVICE;
  return ok(hipStreamWaitEvent(s, t->ev_out_done, 0)) ? HSA_OK : HSA_ERR_DEVICE;
}

// Marks the listed pages (host int32 [batch, n]) in `mark`; errors for
// indices outside the table and pages never placed.
hsa_status_t list_pages(const hsa_tier* t, const int32_t* pages, int32_t n, std::vector<char>& mark) {
  for (int b = 0; b < t->batch; ++b)
    for (int i = 0; i < n; ++i) {
      const int p = pages[(size_t)b * n + i];
      if (p < 0) continue;
      if (p >= t->max_pages) return HSA_ERR_OUT_OF_RANGE;
      const int g = b * t->max_pages + p;
      if (t->loc[g] == -1) return HSA_ERR_INVALID_ARG;   // never placed
      mark[g] = 1;
    }
  return HSA_OK;
}

// Brings every page marked in `want` into L1 on s; pages marked in `pinned`
// (want among them) may not move. UNSUPPORTED, before any move, when the
// pinned pages outnumber the L1 slots.
hsa_status_t bring_all(hsa_tier* t, const std::vector<char>& want, const std::vector<char>& pinned,
                       hipStream_t s) {
  int need = 0;
  for (size_t g = 0; g < pinned.size(); ++g) need += pinned[g] && (want[g] || t->loc[g] >= 0);
  if (need > t->l1_slots) return HSA_ERR_UNSUPPORTED;
  const uint64_t use = ++t->now;
  for (size_t g = 0; g < want.size(); ++g) {
    if (!want[g]) continue;
    t->tick[g] = use;
    const hsa_status_t st = bring(t, (int)g, pinned, s);
    if (st != HSA_OK) return st;
  }
  return HSA_OK;
}

void destroy(hsa_tier* t) {
  if (live(t)) {
    if (t->out_stream) {
      hipStreamSynchronize(t->out_stream);
      hipStreamDestroy(t->out_stream);
    }
    drop_events(t->l1_ev);
    drop_events(t->l2_ev);
    drop_events(t->bounce_ev);
    for (hipEvent_t e : {t->ev_start, t->ev_out_done, t->ev_fetch, t->ev_prefetch})
      if (e) {
        hipEventSynchronize(e);
        hipEventDestroy(e);
      }
    for (char* b : t->bounce)
      if (b) hipHostFree(b);
  }
  if (t->fd >= 0) close(t->fd);
  delete t;
}

// An unnamed file in directory dir (gone when closed); a named one removed
// at once where the file system has no unnamed files.
int open_l3(const char* dir) {
  int fd = open(dir, O_TMPFILE | O_RDWR | O_CLOEXEC, 0600);
  if (fd >= 0) return fd;
  std::string path = std::string(dir) + "/hsa_l3_XXXXXX";
  std::vector<char> buf(path.begin(), path.end());
  buf.push_back('\0');
  fd = mkostemp(buf.data(), O_CLOEXEC);
  if (fd >= 0) unlink(buf.data());
  return fd;
}

}  // namespace

extern "C" {

hsa_status_t hsa_tier_create(const hsa_config_t* cfg, const hsa_kv_pool_t* pool, void* host_k,
                             void* host_v, int32_t l2_slots, const char* l3_dir, int32_t l3_slots,
                             hsa_tier_t** out) {
  if (!cfg || !pool || !out) return HSA_ERR_INVALID_ARG;
  *out = nullptr;
  if (cfg->batch < 1 || cfg->num_heads < 1 || cfg->head_dim < 1 || cfg->page_size < 1)
    return HSA_ERR_INVALID_ARG;
  if (pool->num_slots < 1 || pool->max_pages < 1 || l2_slots < 0 || l3_slots < 0)
    return HSA_ERR_INVALID_ARG;
  if (l3_slots > 0 && l2_slots < 1) return HSA_ERR_INVALID_ARG;
  const bool plan_only = pool->k == nullptr;
  if (!plan_only && (!pool->v || !pool->page_table || (l2_slots > 0 && (!host_k || !host_v)) ||
                     (l3_slots > 0 && !l3_dir)))
    return HSA_ERR_INVALID_ARG;
  if ((size_t)cfg->batch * pool->max_pages > (size_t)INT32_MAX) return HSA_ERR_UNSUPPORTED;
  hsa_tier* t = new hsa_tier();
  t->batch = cfg->batch;
  t->max_pages = pool->max_pages;
  t->l1_slots = pool->num_slots;
  t->l2_slots = l2_slots;
  t->l3_slots = l3_slots;
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
  t->held.assign(n, 0);
  t->table.assign(n, -1);
  t->l1_owner.assign(pool->num_slots, -1);
  t->l2_owner.assign(l2_slots, -1);
  t->l3_owner.assign(l3_slots, -1);
  if (!plan_only) {
    hsa_status_t st = HSA_OK;
    if (!ok(hipStreamCreateWithFlags(&t->out_stream, hipStreamNonBlocking))) st = HSA_ERR_DEVICE;
    for (hipEvent_t* e : {&t->ev_start, &t->ev_out_done, &t->ev_fetch, &t->ev_prefetch})
      if (st == HSA_OK && !ok(hipEventCreateWithFlags(e, hipEventDisableTiming))) st = HSA_ERR_DEVICE;
    if (st == HSA_OK) st = make_events(t->l1_ev, t->l1_slots);
    if (st == HSA_OK) st = make_events(t->l2_ev, t->l2_slots);
    if (st == HSA_OK) st = make_events(t->bounce_ev, 2);
    if (st == HSA_OK && l3_slots > 0) {
      t->fd = open_l3(l3_dir);
      if (t->fd < 0) st = HSA_ERR_IO;
      for (char*& b : t->bounce)
        if (st == HSA_OK && !ok(hipHostMalloc((void**)&b, t->k_bytes + t->v_bytes, hipHostMallocDefault)))
          st = HSA_ERR_DEVICE;
    }
    if (st != HSA_OK) {
      destroy(t);
      return st;
    }
  }
  *out = t;
  return HSA_OK;
}

void hsa_tier_destroy(hsa_tier_t* t) {
  if (t) destroy(t);
}

hsa_status_t hsa_tier_place(hsa_tier_t* t, int32_t b, int32_t page, int32_t* slot, void* stream) {
  if (!t || !slot) return HSA_ERR_INVALID_ARG;
  if (b < 0 || b >= t->batch || page < 0 || page >= t->max_pages) return HSA_ERR_OUT_OF_RANGE;
  const int g = b * t->max_pages + page;
  if (t->loc[g] != -1) return HSA_ERR_INVALID_ARG;  // already placed
  // one lower-tier slot always stays free, so that a fetch can move a page
  // out before the page it brings back has left its slot
  const int lower = t->l2_slots + t->l3_slots;
  const int cap = t->l1_slots + (lower > 0 ? lower - 1 : 0);
  if (t->n_placed >= cap) return HSA_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hsa_status_t st = begin(t, s, nullptr);
  if (st != HSA_OK) return st;
  // on the compute stream every earlier kernel is ordered before the move
  const std::vector<char> pinned(t->loc.size(), 0);
  int sl = -1;
  st = take_l1(t, pinned, &sl);
  if (st == HSA_OK) {
    t->l1_owner[sl] = g;
    t->loc[g] = sl;
    ++t->n_placed;
    t->tick[g] = ++t->now;
    t->held[g] = 1;
    t->table[g] = sl;
    *slot = sl;
    st = publish(t, g, s);
  }
  const hsa_status_t st2 = end(t, s);
  return st != HSA_OK ? st : st2;
}

hsa_status_t hsa_tier_fetch(hsa_tier_t* t, const int32_t* pages, int32_t n_per_batch, void* stream) {
  if (!t || (n_per_batch > 0 && !pages) || n_per_batch < 0) return HSA_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<char> want(t->loc.size(), 0);
  hsa_status_t st = list_pages(t, pages, n_per_batch, want);
  if (st != HSA_OK) return st;
  st = begin(t, s, t->prefetch_pending ? t->ev_prefetch : nullptr);
  if (st != HSA_OK) return st;
  t->prefetch_pending = false;
  st = bring_all(t, want, want, s);
  // the listed pages are what the kernels that follow read
  t->held = want;
  const hsa_status_t st2 = end(t, s);
  if (live(t) && ok(hipEventRecord(t->ev_fetch, s))) t->fetch_recorded = true;
  return st != HSA_OK ? st : st2;
}

hsa_status_t hsa_tier_prefetch(hsa_tier_t* t, const int32_t* pages, int32_t n_per_batch, void* stream) {
  if (!t || (n_per_batch > 0 && !pages) || n_per_batch < 0) return HSA_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<char> want(t->loc.size(), 0);
  hsa_status_t st = list_pages(t, pages, n_per_batch, want);
  if (st != HSA_OK) return st;
  // the pages the compute stream's kernels may read stay where they are
  std::vector<char> pinned(t->held);
  for (size_t g = 0; g < want.size(); ++g) pinned[g] |= want[g];
  st = begin(t, s, t->fetch_recorded ? t->ev_fetch : nullptr);
  if (st != HSA_OK) return st;
  const int64_t before = t->stats.fetches;
  st = bring_all(t, want, pinned, s);
  t->stats.prefetched += t->stats.fetches - before;
  hsa_status_t st2 = end(t, s);
  if (live(t)) {
    if (ok(hipEventRecord(t->ev_prefetch, s)))
      t->prefetch_pending = true;
    else if (st2 == HSA_OK)
      st2 = HSA_ERR_DEVICE;
  }
  return st != HSA_OK ? st : st2;
}

int32_t hsa_tier_locate(const hsa_tier_t* t, int32_t b, int32_t page) {
  if (!t || b < 0 || b >= t->batch || page < 0 || page >= t->max_pages) return -1;
  return t->loc[(size_t)b * t->max_pages + page];
}

void hsa_tier_stats(const hsa_tier_t* t, hsa_tier_stats_t* out) {
  if (t && out) *out = t->stats;
}

}  // extern "C"

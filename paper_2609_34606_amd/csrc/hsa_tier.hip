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
// that read the pool. A fetch moves each page with one swap kernel on that
// stream: the incoming page (from a host slot or a staging page) and the
// page it displaces (into the host slot the incoming one leaves) cross the
// link in both directions at once, in place, so a swap needs no free host
// slot. Place and prefetch use DMA copies, which take no compute units:
// host-to-device on the calling stream, device-to-host (pages leaving L1) on
// an internal stream. A prefetch runs on a side stream of the
// caller's: its copies overlap the kernels of the compute stream, it never
// moves a page the kernels may read (those of the last fetch and pages placed
// since), it starts after the compute stream has passed the last fetch, and
// the next fetch waits for it. Every async copy records an event on the
// block it touches (the key or value block of a pool slot, host slot or
// staging buffer); the next copy or host access of that block waits for it,
// so copies issued on different streams never overlap on one block. A page
// a DMA copy moves out takes the free host slot freed first, so that it does
// not wait for a page that just came in through the same slot. Page-table
// updates of a fetch are written by one small kernel at the end of the
// call. Without device pointers ("plan-only") the same bookkeeping runs and
// no copy, event or file access is issued.
//
// Backup mode. The file then holds a copy of every page: each page owns a
// file slot from its placement on, is written there by the first commit
// after the caller has written it (or when it leaves L1 and L2 before that
// commit), and keeps it. A page leaving L2 whose copy is written costs no
// file write, a read from L3 leaves the file copy in place, and dropping
// every L1 and L2 copy leaves each page restorable from the file.
#include <errno.h>
#include <fcntl.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <algorithm>
#include <memory>
#include <string>
#include <vector>

#include "hsa_kernels.h"

namespace {

// Events recorded after async copies and launches. One event serves every
// block that copy or launch touched, and goes back to the pool's free list
// once no block refers to it (nothing can wait for that record any more).
struct EvPool {
  std::vector<hipEvent_t> all, free;
};
struct EvBox {
  hipEvent_t ev;
  hipStream_t by;   // the stream it was recorded on
  EvPool* pool;
  ~EvBox() { pool->free.push_back(ev); }
};
using EvRef = std::shared_ptr<EvBox>;

// Per slot, the event of the last async copy of each of its two blocks (key
// block, value block): a copy into one block waits only for the copies of
// that block.
constexpr int kParts = 2;
struct SlotEvents {
  std::vector<EvRef> ev;        // [slot * kParts + part]; null: no copy yet
  std::vector<char> pending;    // touched by the queued swap launch, event not yet recorded
  hsa_tier* owner = nullptr;
};

// A swap of one block of a pool slot with host memory, in place: each
// element of the slot is read (for `out`) and the incoming element read (from
// `in`) before either is written, so `out` may be the very host block `in`
// names. in == NULL: only the slot's content goes out; out == NULL: only
// `in` comes in. Host addresses are device addresses of pinned host memory.
struct SwapBlock {
  char* dev;
  const char* in;
  char* out;
  uint64_t n16;   // 16-byte elements
};
constexpr int kSwapMax = 16;      // blocks per launch (8 pages)
constexpr int kSwapGroups = 16;   // workgroups per block: with 8+ blocks, enough requests in flight
struct SwapArgs {
  SwapBlock blk[kSwapMax];
};

hsa_status_t flush_swaps(hsa_tier* t);

}  // namespace

struct hsa_tier {
  int32_t batch, max_pages, l1_slots, l2_slots, l3_slots;
  int32_t n_placed = 0;
  bool backup = false;       // the file holds a copy of every page
  size_t k_bytes, v_bytes;   // bytes of one slot of the key / value pool
  char* dev_k;               // device pool (NULL: plan-only)
  char* dev_v;
  int32_t* dev_table;        // device page table [batch, max_pages]
  char* host_k;              // pinned host slots (L2)
  char* host_v;
  char* host_k_dev = nullptr;     // the same host memory as the device addresses it
  char* host_v_dev = nullptr;
  char* bounce_dev[2] = {nullptr, nullptr};
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
  std::vector<uint64_t> l2_freed;  // per host slot: when it was last freed
  std::vector<int32_t> bak;        // backup mode: file slot of each page, or -1
  std::vector<char> backed;        // backup mode: that file slot holds the page
  std::vector<int32_t> pub;        // page indices whose table entry changed
  uint64_t now = 0, frees = 0;
  hsa_tier_stats_t stats{};
  // live mode only
  hipStream_t out_stream = nullptr;        // device-to-host copies
  EvPool evpool;
  SlotEvents l1_ev, l2_ev, bounce_ev;
  // the swaps a fetch queues, issued as one launch on swap_stream, and the
  // block events to record after it
  std::vector<SwapBlock> swaps;
  std::vector<std::pair<SlotEvents*, size_t>> swap_marks;
  hipStream_t swap_stream = nullptr;
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

void make_events(hsa_tier* t, SlotEvents& e, int n) {
  e.owner = t;
  e.ev.assign((size_t)n * kParts, nullptr);
  e.pending.assign((size_t)n * kParts, 0);
}

// An event recorded on s now.
hsa_status_t record(hsa_tier* t, hipStream_t s, EvRef* out) {
  EvPool& p = t->evpool;
  if (p.free.empty()) {
    hipEvent_t e = nullptr;
    if (!ok(hipEventCreateWithFlags(&e, hipEventDisableTiming))) return HSA_ERR_DEVICE;
    p.all.push_back(e);
    p.free.push_back(e);
  }
  hipEvent_t e = p.free.back();
  p.free.pop_back();
  *out = EvRef(new EvBox{e, s, &p});
  return ok(hipEventRecord(e, s)) ? HSA_OK : HSA_ERR_DEVICE;
}

// Waits for every event, then destroys them (no block may refer to one).
void drop_events(EvPool& p) {
  for (hipEvent_t e : p.all) {
    hipEventSynchronize(e);
    hipEventDestroy(e);
  }
  p.all.clear();
  p.free.clear();
}

// A block the queued swap launch touches has no event yet: issue the launch
// (and record its event) before anything waits for that block.
hsa_status_t settle(SlotEvents& e, size_t x) {
  return e.pending[x] ? flush_swaps(e.owner) : HSA_OK;
}

// Stream s waits for the last copy on block `part` of slot i (nothing to do
// when that copy was issued on s itself).
hsa_status_t after(hipStream_t s, SlotEvents& e, int i, int part) {
  const size_t x = (size_t)i * kParts + part;
  hsa_status_t st = settle(e, x);
  const EvBox* b = e.ev[x].get();
  if (st != HSA_OK || !b || b->by == s) return st;
  return ok(hipStreamWaitEvent(s, b->ev, 0)) ? HSA_OK : HSA_ERR_DEVICE;
}

// The host waits for the last copies on slot i (before reading or writing it).
hsa_status_t host_wait(SlotEvents& e, int i) {
  for (int part = 0; part < kParts; ++part) {
    const size_t x = (size_t)i * kParts + part;
    const hsa_status_t st = settle(e, x);
    if (st != HSA_OK) return st;
    if (e.ev[x] && !ok(hipEventSynchronize(e.ev[x]->ev))) return HSA_ERR_DEVICE;
  }
  return HSA_OK;
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

// One page (key block dk <- sk, value block dv <- sv) copied on s, block by
// block: each block's copy waits for the last copies of that block in the
// destination slot (ed, id) and the source slot (es, is) and is recorded on
// both.
hsa_status_t page_copy(hsa_tier* t, hipStream_t s, hipMemcpyKind kind, char* dk, char* dv,
                       const char* sk, const char* sv, SlotEvents& ed, int id, SlotEvents& es,
                       int is) {
  hsa_status_t st = HSA_OK;
  for (int part = 0; part < kParts && st == HSA_OK; ++part) {
    st = after(s, ed, id, part);
    if (st == HSA_OK) st = after(s, es, is, part);
    if (st == HSA_OK)
      st = part == 0 ? copy(dk, sk, t->k_bytes, kind, s) : copy(dv, sv, t->v_bytes, kind, s);
    EvRef r;
    if (st == HSA_OK) st = record(t, s, &r);
    if (st == HSA_OK) ed.ev[(size_t)id * kParts + part] = es.ev[(size_t)is * kParts + part] = r;
  }
  return st;
}

__global__ __launch_bounds__(256) void swap_kernel(SwapArgs a) {
  const SwapBlock b = a.blk[blockIdx.y];
  uint4* dev = reinterpret_cast<uint4*>(b.dev);
  const uint4* in = reinterpret_cast<const uint4*>(b.in);
  uint4* out = reinterpret_cast<uint4*>(b.out);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < b.n16; i += stride) {
    uint4 x{}, y{};
    if (out) x = dev[i];
    if (in) y = in[i];
    if (out) out[i] = x;
    if (in) dev[i] = y;
  }
}

// Queues the swap of pool slot sl with host memory on s: the slot's page
// goes to L2 slot `a` (a < 0: nowhere), the page at in_k / in_v (device
// addresses; NULL: none) comes in. The stream first waits for the last
// copies of the slot's blocks, the source's (ein, iin) and L2 slot a's; the
// events of all of them are recorded after the launch (flush_swaps).
hsa_status_t swap_page(hsa_tier* t, hipStream_t s, int sl, const char* in_k, const char* in_v,
                       SlotEvents* ein, int iin, int a) {
  hsa_status_t st = HSA_OK;
  if (t->swaps.size() + kParts > (size_t)kSwapMax || (t->swap_stream && t->swap_stream != s))
    st = flush_swaps(t);
  for (int part = 0; part < kParts && st == HSA_OK; ++part) {
    st = after(s, t->l1_ev, sl, part);
    if (st == HSA_OK && ein) st = after(s, *ein, iin, part);
    if (st == HSA_OK && a >= 0 && !(ein == &t->l2_ev && iin == a)) st = after(s, t->l2_ev, a, part);
  }
  if (st != HSA_OK) return st;
  t->swap_stream = s;
  t->swaps.push_back({t->dev_k + (size_t)sl * t->k_bytes, in_k,
                      a >= 0 ? t->host_k_dev + (size_t)a * t->k_bytes : nullptr, t->k_bytes / 16});
  t->swaps.push_back({t->dev_v + (size_t)sl * t->v_bytes, in_v,
                      a >= 0 ? t->host_v_dev + (size_t)a * t->v_bytes : nullptr, t->v_bytes / 16});
  auto defer = [&](SlotEvents& e, int i) {
    for (int part = 0; part < kParts; ++part) {
      const size_t x = (size_t)i * kParts + part;
      if (!e.pending[x]) t->swap_marks.push_back({&e, x});
      e.pending[x] = 1;
    }
  };
  defer(t->l1_ev, sl);
  if (ein) defer(*ein, iin);
  if (a >= 0) defer(t->l2_ev, a);
  return HSA_OK;
}

// Issues the queued swaps as one launch and records the events of the
// blocks they touch.
hsa_status_t flush_swaps(hsa_tier* t) {
  if (t->swaps.empty()) return HSA_OK;
  SwapArgs args;
  const int n = (int)t->swaps.size();
  for (int i = 0; i < n; ++i) args.blk[i] = t->swaps[i];
  t->swaps.clear();
  hipStream_t s = t->swap_stream;
  t->swap_stream = nullptr;
  swap_kernel<<<dim3(kSwapGroups, n), 256, 0, s>>>(args);
  hsa_status_t st = ok(hipGetLastError()) ? HSA_OK : HSA_ERR_DEVICE;
  EvRef r;
  if (st == HSA_OK) st = record(t, s, &r);
  for (auto& m : t->swap_marks) {
    m.first->pending[m.second] = 0;
    m.first->ev[m.second] = r;
  }
  t->swap_marks.clear();
  return st;
}

// Page-table entries, passed by value (a copy from host memory that later
// calls change could run after the change).
constexpr int kTableWrites = 64;
struct TableWrites {
  int32_t n;
  int32_t idx[kTableWrites];
  int32_t val[kTableWrites];
};

__global__ void set_entries_kernel(int32_t* table, TableWrites w) {
  const int i = threadIdx.x;
  if (i < w.n) table[w.idx[i]] = w.val[i];
}

// Writes the entries of the pages queued in t->pub to the device page table
// on s, in launches of up to kTableWrites entries.
hsa_status_t publish(hsa_tier* t, hipStream_t s) {
  if (!live(t)) {
    t->pub.clear();
    return HSA_OK;
  }
  for (size_t i = 0; i < t->pub.size(); i += kTableWrites) {
    TableWrites w;
    w.n = (int32_t)std::min<size_t>(kTableWrites, t->pub.size() - i);
    for (int j = 0; j < w.n; ++j) {
      w.idx[j] = t->pub[i + j];
      w.val[j] = t->table[t->pub[i + j]];
    }
    set_entries_kernel<<<1, kTableWrites, 0, s>>>(t->dev_table, w);
    if (!ok(hipGetLastError())) return HSA_ERR_DEVICE;
  }
  t->pub.clear();
  return HSA_OK;
}

// A free L3 slot, or -1 (a page's own slot in backup mode is never free).
int free_l3(const hsa_tier* t) {
  for (int i = 0; i < t->l3_slots; ++i)
    if (t->l3_owner[i] < 0) return i;
  return -1;
}

// The free L2 slot freed first, or -1.
int free_l2(const hsa_tier* t) {
  int best = -1;
  for (int i = 0; i < t->l2_slots; ++i)
    if (t->l2_owner[i] < 0 && (best < 0 || t->l2_freed[i] < t->l2_freed[best])) best = i;
  return best;
}

void release_l2(hsa_tier* t, int i) {
  t->l2_owner[i] = -1;
  t->l2_freed[i] = ++t->frees;
}

// Writes host bytes (key block k, value block v) of page g to file slot c.
hsa_status_t write_slot(hsa_tier* t, const char* k, const char* v, int c) {
  hsa_status_t st = file_io(t->fd, const_cast<char*>(k), t->k_bytes, l3_offset(t, c), true);
  if (st == HSA_OK)
    st = file_io(t->fd, const_cast<char*>(v), t->v_bytes, l3_offset(t, c) + (off_t)t->k_bytes, true);
  return st;
}

// The file slot page g goes to when it leaves L2 (or L1 straight to L3):
// its own slot in backup mode, else a free one (-1: none).
int l3_target(const hsa_tier* t, int g) { return t->backup ? t->bak[g] : free_l3(t); }

// Whether moving page g to L3 writes the file (not when its backup is there).
bool needs_write(const hsa_tier* t, int g) { return !t->backup || !t->backed[g]; }

void count_write(hsa_tier* t, int g) {
  if (!t->backup) return;
  t->backed[g] = 1;
  ++t->stats.backups;
}

// A free L2 slot; when none is free, the least recently used L2 page that is
// not pinned moves to L3 first (written from its host slot after the copy
// that filled it, unless its backup is already in the file).
hsa_status_t take_l2(hsa_tier* t, const std::vector<char>& pinned, int* out) {
  const int f = free_l2(t);
  if (f >= 0) {
    *out = f;
    return HSA_OK;
  }
  int w = -1;
  for (int i = 0; i < t->l2_slots; ++i) {
    const int g = t->l2_owner[i];
    if (pinned[g]) continue;
    if (w < 0 || t->tick[g] < t->tick[t->l2_owner[w]]) w = i;
  }
  if (w < 0) return HSA_ERR_UNSUPPORTED;   // every L2 page is needed now (or no L2)
  const int g = t->l2_owner[w];
  const int c = l3_target(t, g);
  if (c < 0) return HSA_ERR_UNSUPPORTED;   // every tier is full
  if (needs_write(t, g)) {
    if (live(t)) {
      hsa_status_t st = host_wait(t->l2_ev, w);
      if (st == HSA_OK)
        st = write_slot(t, t->host_k + (size_t)w * t->k_bytes, t->host_v + (size_t)w * t->v_bytes, c);
      if (st != HSA_OK) return st;
    }
    count_write(t, g);
  }
  t->l3_owner[c] = g;
  release_l2(t, w);
  t->loc[g] = l3_code(t, c);
  ++t->stats.spills;
  *out = w;
  return HSA_OK;
}

// Copies L1 slot v into staging page j on the internal stream (after the
// last copy on either).
hsa_status_t stage_out(hsa_tier* t, int v, int j) {
  return page_copy(t, t->out_stream, hipMemcpyDeviceToHost, t->bounce[j], t->bounce[j] + t->k_bytes,
                   t->dev_k + (size_t)v * t->k_bytes, t->dev_v + (size_t)v * t->v_bytes,
                   t->bounce_ev, j, t->l1_ev, v);
}

// Moves the page in L1 slot v straight to L3 slot c through a staging page
// (when no L2 slot can take it); no copy when its backup is in the file.
hsa_status_t l1_to_l3(hsa_tier* t, int v, int c) {
  const int g = t->l1_owner[v];
  if (!needs_write(t, g)) return HSA_OK;
  if (live(t)) {
    const int j = t->next_bounce;
    t->next_bounce ^= 1;
    hsa_status_t st = stage_out(t, v, j);
    if (st == HSA_OK) st = host_wait(t->bounce_ev, j);
    if (st == HSA_OK) st = write_slot(t, t->bounce[j], t->bounce[j] + t->k_bytes, c);
    if (st != HSA_OK) return st;
  }
  count_write(t, g);
  return HSA_OK;
}

// A free L1 slot, moving the least recently used unpinned resident page down
// a tier first when none is free: to L2, or to L3 when no L2 page may make
// room. The page going to L2 takes host slot `prefer` when given (the slot
// the incoming page leaves in the same swap), else a free one. With `defer`
// its device-to-host copy is left to the caller (*defer_a = its L2 slot);
// else it is issued on the internal stream. Fails before changing anything
// when no page may move.
hsa_status_t take_l1(hsa_tier* t, const std::vector<char>& pinned, int prefer, bool defer, int* out,
                     int* defer_a) {
  *defer_a = -1;
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
  int a = prefer;
  hsa_status_t st = prefer >= 0 ? HSA_OK : take_l2(t, pinned, &a);
  if (st == HSA_ERR_UNSUPPORTED) {
    const int c = l3_target(t, g);
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
  if (defer) {
    *defer_a = a;
  } else if (live(t)) {
    st = page_copy(t, t->out_stream, hipMemcpyDeviceToHost, t->host_k + (size_t)a * t->k_bytes,
                   t->host_v + (size_t)a * t->v_bytes, t->dev_k + (size_t)v * t->k_bytes,
                   t->dev_v + (size_t)v * t->v_bytes, t->l2_ev, a, t->l1_ev, v);
    if (st != HSA_OK) return st;
  }
  t->l2_owner[a] = g;
  t->l1_owner[v] = -1;
  t->loc[g] = l2_code(a);
  ++t->stats.evictions;
  *out = v;
  return HSA_OK;
}

// Brings page index g into L1 on s; its page-table entry is queued for
// publish(). With `swap` (a fetch) one swap kernel moves the page in and
// the page it displaces out, the latter into the host slot the former
// leaves; else (a prefetch) DMA copies: the displaced page on the internal
// stream, the incoming one on s.
hsa_status_t bring(hsa_tier* t, int g, const std::vector<char>& pinned, hipStream_t s, bool swap) {
  const int loc = t->loc[g];
  if (loc >= 0) return HSA_OK;
  const int i2 = l2_index(t, loc), i3 = l3_index(t, loc);
  int sl = -1, j = -1, a = -1;
  hsa_status_t st;
  if (i3 >= 0) {
    // read into a staging buffer first: the L3 slot is then free for a spill
    // that making room in L1 may cause (in backup mode it stays the page's)
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
    if (!t->backup) t->l3_owner[i3] = -1;
    st = take_l1(t, pinned, -1, swap, &sl, &a);
    if (st != HSA_OK) {
      t->l3_owner[i3] = g;   // nothing was written over it
      return st;
    }
    ++t->stats.reloads;
  } else {
    st = take_l1(t, pinned, swap ? i2 : -1, swap, &sl, &a);
    if (st != HSA_OK) return st;
  }
  if (live(t)) {
    if (swap) {
      const char* sk = i3 >= 0 ? t->bounce_dev[j] : t->host_k_dev + (size_t)i2 * t->k_bytes;
      const char* sv = i3 >= 0 ? t->bounce_dev[j] + t->k_bytes : t->host_v_dev + (size_t)i2 * t->v_bytes;
      st = swap_page(t, s, sl, sk, sv, i3 >= 0 ? &t->bounce_ev : &t->l2_ev, i3 >= 0 ? j : i2, a);
    } else {
      const char* sk = i3 >= 0 ? t->bounce[j] : t->host_k + (size_t)i2 * t->k_bytes;
      const char* sv = i3 >= 0 ? t->bounce[j] + t->k_bytes : t->host_v + (size_t)i2 * t->v_bytes;
      st = page_copy(t, s, hipMemcpyHostToDevice, t->dev_k + (size_t)sl * t->k_bytes,
                     t->dev_v + (size_t)sl * t->v_bytes, sk, sv, t->l1_ev, sl,
                     i3 >= 0 ? t->bounce_ev : t->l2_ev, i3 >= 0 ? j : i2);
    }
    if (st != HSA_OK) return st;
  }
  // the host slot the page came from, unless the displaced page took it
  if (i2 >= 0 && t->l2_owner[i2] == g) release_l2(t, i2);
  t->l1_owner[sl] = g;
  t->loc[g] = sl;
  t->table[g] = sl;
  t->pub.push_back(g);
  ++t->stats.fetches;
  return HSA_OK;
}

// Orders a call's copies after the work already on s (and after `wait`, if
// given): the internal stream starts where s is now.
hsa_status_t begin(hsa_tier* t, hipStream_t s, hipEvent_t wait) {
  if (!live(t)) return HSA_OK;
  if (wait && !ok(hipStreamWaitEvent(s, wait, 0))) return HSA_ERR_DEVICE;
  if (!ok(hipEventRecord(t->ev_start, s))) return HSA_ERR_DEVICE;
  return ok(hipStreamWaitEvent(t->out_stream, t->ev_start, 0)) ? HSA_OK : HSA_ERR_DEVICE;
}

// Publishes the queued page-table entries on s; work issued on s after the
// call starts after all of the call's copies.
hsa_status_t end(hsa_tier* t, hipStream_t s) {
  const hsa_status_t st = publish(t, s);
  if (!live(t)) return st;
  if (!ok(hipEventRecord(t->ev_out_done, t->out_stream))) return HSA_ERR_DEVICE;
  if (!ok(hipStreamWaitEvent(s, t->ev_out_done, 0))) return HSA_ERR_DEVICE;
  return st;
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
                       hipStream_t s, bool swap) {
  int need = 0;
  for (size_t g = 0; g < pinned.size(); ++g) need += pinned[g] && (want[g] || t->loc[g] >= 0);
  if (need > t->l1_slots) return HSA_ERR_UNSUPPORTED;
  const uint64_t use = ++t->now;
  for (size_t g = 0; g < want.size(); ++g) {
    if (!want[g]) continue;
    t->tick[g] = use;
    const hsa_status_t st = bring(t, (int)g, pinned, s, swap);
    if (st != HSA_OK) return st;
  }
  return HSA_OK;
}

// Backup mode: writes every placed page whose file copy is not written yet,
// after the work already on s (the caller's writes of the page). Pages in
// L1 go through the two staging pages, the copy of the next page running
// while the host writes the current one; pages in L2 are written from their
// host slot. Blocks until the file writes are issued (pwrite).
hsa_status_t commit_all(hsa_tier* t, hipStream_t s) {
  std::vector<int> todo;
  for (size_t g = 0; g < t->loc.size(); ++g)
    if (t->loc[g] != -1 && !t->backed[g]) todo.push_back((int)g);
  if (todo.empty() || !live(t)) {
    for (int g : todo) count_write(t, g);
    return HSA_OK;
  }
  hsa_status_t st = begin(t, s, nullptr);
  // stage(i): the staging page of todo[i] once its copy is issued (-1: not
  // staged, the page is in L2)
  std::vector<int> staged(todo.size(), -1);
  auto stage = [&](size_t i) -> hsa_status_t {
    const int loc = t->loc[todo[i]];
    if (loc < 0) return HSA_OK;
    const int j = t->next_bounce;
    t->next_bounce ^= 1;
    staged[i] = j;
    return stage_out(t, loc, j);
  };
  if (st == HSA_OK) st = stage(0);
  for (size_t i = 0; i < todo.size() && st == HSA_OK; ++i) {
    if (i + 1 < todo.size()) st = stage(i + 1);
    if (st != HSA_OK) break;
    const int g = todo[i];
    const int c = t->bak[g];
    const int j = staged[i];
    if (j >= 0) {
      st = host_wait(t->bounce_ev, j);
      if (st == HSA_OK) st = write_slot(t, t->bounce[j], t->bounce[j] + t->k_bytes, c);
    } else {
      const int a = l2_index(t, t->loc[g]);
      st = host_wait(t->l2_ev, a);
      if (st == HSA_OK)
        st = write_slot(t, t->host_k + (size_t)a * t->k_bytes, t->host_v + (size_t)a * t->v_bytes, c);
    }
    if (st == HSA_OK) count_write(t, g);
  }
  const hsa_status_t st2 = end(t, s);
  return st != HSA_OK ? st : st2;
}

void destroy(hsa_tier* t) {
  if (live(t)) {
    flush_swaps(t);
    if (t->out_stream) {
      hipStreamSynchronize(t->out_stream);
      hipStreamDestroy(t->out_stream);
    }
    for (SlotEvents* e : {&t->l1_ev, &t->l2_ev, &t->bounce_ev}) e->ev.clear();
    drop_events(t->evpool);
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
                             int32_t l3_backup, hsa_tier_t** out) {
  if (!cfg || !pool || !out) return HSA_ERR_INVALID_ARG;
  *out = nullptr;
  if (cfg->batch < 1 || cfg->num_heads < 1 || cfg->head_dim < 1 || cfg->page_size < 1)
    return HSA_ERR_INVALID_ARG;
  if (pool->num_slots < 1 || pool->max_pages < 1 || l2_slots < 0 || l3_slots < 0)
    return HSA_ERR_INVALID_ARG;
  if (l3_backup ? l3_slots < 1 : (l3_slots > 0 && l2_slots < 1)) return HSA_ERR_INVALID_ARG;
  const bool plan_only = pool->k == nullptr;
  if (!plan_only && (!pool->v || !pool->page_table || (l2_slots > 0 && (!host_k || !host_v)) ||
                     (l3_slots > 0 && !l3_dir)))
    return HSA_ERR_INVALID_ARG;
  if ((size_t)cfg->batch * pool->max_pages > (size_t)INT32_MAX) return HSA_ERR_UNSUPPORTED;
  // the swap kernel moves 16-byte elements: slot blocks and bases 16-byte aligned
  const size_t block_bytes =
      (size_t)cfg->num_heads * cfg->page_size * cfg->head_dim * (cfg->dtype == HSA_DTYPE_BF16 ? 2 : 4);
  auto misaligned = [](const void* p) { return ((uintptr_t)p & 15) != 0; };
  if (block_bytes % 16 || misaligned(pool->k) || misaligned(pool->v) || misaligned(host_k) ||
      misaligned(host_v))
    return HSA_ERR_UNSUPPORTED;
  hsa_tier* t = new hsa_tier();
  t->batch = cfg->batch;
  t->max_pages = pool->max_pages;
  t->l1_slots = pool->num_slots;
  t->l2_slots = l2_slots;
  t->l3_slots = l3_slots;
  t->backup = l3_backup != 0;
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
  t->l2_freed.assign(l2_slots, 0);
  if (t->backup) {
    t->bak.assign(n, -1);
    t->backed.assign(n, 0);
  }
  if (!plan_only) {
    hsa_status_t st = HSA_OK;
    if (!ok(hipStreamCreateWithFlags(&t->out_stream, hipStreamNonBlocking))) st = HSA_ERR_DEVICE;
    for (hipEvent_t* e : {&t->ev_start, &t->ev_out_done, &t->ev_fetch, &t->ev_prefetch})
      if (st == HSA_OK && !ok(hipEventCreateWithFlags(e, hipEventDisableTiming))) st = HSA_ERR_DEVICE;
    make_events(t, t->l1_ev, t->l1_slots);
    make_events(t, t->l2_ev, t->l2_slots);
    make_events(t, t->bounce_ev, 2);
    // the swap kernel addresses the host slots and staging pages directly
    if (st == HSA_OK && l2_slots > 0 &&
        (!ok(hipHostGetDevicePointer((void**)&t->host_k_dev, host_k, 0)) ||
         !ok(hipHostGetDevicePointer((void**)&t->host_v_dev, host_v, 0))))
      st = HSA_ERR_INVALID_ARG;   // not pinned host memory
    if (st == HSA_OK && l3_slots > 0) {
      t->fd = open_l3(l3_dir);
      if (t->fd < 0) st = HSA_ERR_IO;
      for (int j = 0; j < 2 && st == HSA_OK; ++j) {
        if (!ok(hipHostMalloc((void**)&t->bounce[j], t->k_bytes + t->v_bytes, hipHostMallocDefault)) ||
            !ok(hipHostGetDevicePointer((void**)&t->bounce_dev[j], t->bounce[j], 0)))
          st = HSA_ERR_DEVICE;
      }
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
  // out before the page it brings back has left its slot; in backup mode
  // every page owns a file slot instead
  const int lower = t->l2_slots + t->l3_slots;
  const int cap = t->backup ? t->l3_slots : t->l1_slots + (lower > 0 ? lower - 1 : 0);
  if (t->n_placed >= cap) return HSA_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hsa_status_t st = begin(t, s, nullptr);
  if (st != HSA_OK) return st;
  // on the compute stream every earlier kernel is ordered before the move
  const std::vector<char> pinned(t->loc.size(), 0);
  int sl = -1, unused = -1;
  st = take_l1(t, pinned, -1, false, &sl, &unused);
  if (st == HSA_OK) {
    if (t->backup) {
      t->bak[g] = t->n_placed;   // file slots are handed out in placement order
      t->l3_owner[t->n_placed] = g;
    }
    t->l1_owner[sl] = g;
    t->loc[g] = sl;
    ++t->n_placed;
    t->tick[g] = ++t->now;
    t->held[g] = 1;
    t->table[g] = sl;
    t->pub.push_back(g);
    *slot = sl;
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
  st = bring_all(t, want, want, s, true);
  // the moves made so far, also when one failed
  const hsa_status_t st1 = flush_swaps(t);
  if (st == HSA_OK) st = st1;
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
  st = bring_all(t, want, pinned, s, false);
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

hsa_status_t hsa_tier_commit(hsa_tier_t* t, void* stream) {
  if (!t || !t->backup) return HSA_ERR_INVALID_ARG;
  return commit_all(t, static_cast<hipStream_t>(stream));
}

hsa_status_t hsa_tier_drop(hsa_tier_t* t, void* stream) {
  if (!t || !t->backup) return HSA_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hsa_status_t st = commit_all(t, s);
  if (st != HSA_OK) return st;
  st = begin(t, s, t->prefetch_pending ? t->ev_prefetch : nullptr);
  if (st != HSA_OK) return st;
  t->prefetch_pending = false;
  for (size_t g = 0; g < t->loc.size(); ++g) {
    const int loc = t->loc[g];
    if (loc == -1) continue;
    if (loc >= 0)
      t->l1_owner[loc] = -1;
    else if (l2_index(t, loc) >= 0)
      release_l2(t, l2_index(t, loc));
    t->loc[g] = l3_code(t, t->bak[g]);
    // entries of pages that left the pool earlier still name their old slot
    if (t->table[g] != -1) {
      t->table[g] = -1;
      t->pub.push_back((int)g);
    }
  }
  std::fill(t->held.begin(), t->held.end(), 0);
  st = end(t, s);
  // a later prefetch starts after the kernels issued before the drop
  if (live(t) && ok(hipEventRecord(t->ev_fetch, s))) t->fetch_recorded = true;
  return st;
}

int32_t hsa_tier_locate(const hsa_tier_t* t, int32_t b, int32_t page) {
  if (!t || b < 0 || b >= t->batch || page < 0 || page >= t->max_pages) return -1;
  return t->loc[(size_t)b * t->max_pages + page];
}

void hsa_tier_stats(const hsa_tier_t* t, hsa_tier_stats_t* out) {
  if (t && out) *out = t->stats;
}

}  // extern "C"

// C ABI of the HSA library: argument validation, launch planning and
// workspace layout. Every computation happens in the kernels; this file only
// checks arguments, sizes the grids and hands pointers over.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "hsa_kernels.h"

using namespace hsa;

namespace {

constexpr size_t kAlign = 256;
constexpr int kStateTargetGroups = 512;  // ~2 workgroups per CU on 256 CUs
constexpr int kQsumRows = 32;
constexpr int kPartPerHead = 4;  // partial slots per head for split key lists
constexpr int kPageWaves = 8;    // attention workgroup width for the page walk

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool check_env() {
  const char* e = getenv("HSA_CHECK");
  return e && e[0] == '1';
}

hsa_status_t check_cfg(const hsa_config_t* c) {
  if (!c) return HSA_ERR_INVALID_ARG;
  if (c->batch < 1 || c->num_heads < 1 || c->head_dim < 1 || c->page_size < 1)
    return HSA_ERR_INVALID_ARG;
  if (c->dtype != HSA_DTYPE_BF16 && c->dtype != HSA_DTYPE_F32) return HSA_ERR_UNSUPPORTED;
  if (c->num_heads > HSA_MAX_HEADS) return HSA_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return HSA_ERR_UNSUPPORTED;
  if (c->page_size < 8 || c->page_size % 8 != 0) return HSA_ERR_UNSUPPORTED;
  if (!(c->sm_scale >= 0.f) || isinf(c->sm_scale)) return HSA_ERR_INVALID_ARG;
  if (c->gate_dims != 0 && c->gate_dims != 1 && c->gate_dims != c->head_dim)
    return HSA_ERR_INVALID_ARG;
  return HSA_OK;
}

hsa_status_t check_pool(const hsa_kv_pool_t* p) {
  if (!p || !p->k || !p->v || !p->page_table) return HSA_ERR_INVALID_ARG;
  if (p->num_slots < 1 || p->max_pages < 1) return HSA_ERR_INVALID_ARG;
  return HSA_OK;
}

// With HSA_CHECK=1: every page table entry in [first, first+n) must name a
// slot of the pool.
hsa_status_t validate_pages(const hsa_config_t* c, const hsa_kv_pool_t* p, int first, int n,
                            hipStream_t s) {
  if (!check_env() || n <= 0) return HSA_OK;
  std::vector<int32_t> pt((size_t)c->batch * p->max_pages);
  if (hipStreamSynchronize(s) != hipSuccess) return HSA_ERR_DEVICE;
  if (hipMemcpy(pt.data(), p->page_table, pt.size() * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return HSA_ERR_DEVICE;
  for (int b = 0; b < c->batch; ++b)
    for (int i = first; i < first + n; ++i) {
      const int32_t slot = pt[(size_t)b * p->max_pages + i];
      if (slot < 0 || slot >= p->num_slots) return HSA_ERR_OUT_OF_RANGE;
    }
  return HSA_OK;
}

// With HSA_CHECK=1: every selected page (entries up to the first one outside
// [0, max_pages), as the kernels read them) must map to a slot of the pool.
hsa_status_t validate_selection(const hsa_config_t* c, const hsa_kv_pool_t* p,
                                const int32_t* sel, int k_max, hipStream_t s) {
  if (!check_env() || k_max <= 0) return HSA_OK;
  const size_t rows = (size_t)c->batch * c->num_heads;
  std::vector<int32_t> sl(rows * k_max), pt((size_t)c->batch * p->max_pages);
  if (hipStreamSynchronize(s) != hipSuccess) return HSA_ERR_DEVICE;
  if (hipMemcpy(sl.data(), sel, sl.size() * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(pt.data(), p->page_table, pt.size() * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return HSA_ERR_DEVICE;
  for (size_t r = 0; r < rows; ++r) {
    const size_t b = r / c->num_heads;
    for (int i = 0; i < k_max; ++i) {
      const int32_t e = sl[r * k_max + i];
      if (e < 0 || e >= p->max_pages) break;
      const int32_t slot = pt[b * p->max_pages + e];
      if (slot < 0 || slot >= p->num_slots) return HSA_ERR_OUT_OF_RANGE;
    }
  }
  return HSA_OK;
}

float softmax_scale(const hsa_config_t* c) {
  return c->sm_scale > 0.f ? c->sm_scale : 1.f / sqrtf((float)c->head_dim);
}

struct StatePlan {
  int parts, part_len, upw, n_groups;
};

StatePlan plan_state(const hsa_config_t* c, int n_pages) {
  // A unit is one of `parts` equal key ranges of a page; each workgroup
  // folds upw consecutive units. The pass runs two workgroups per CU, i.e.
  // rounds of kStateTargetGroups; the cost model (in 64-key tiles per slot)
  // counts whole rounds, a fixed cost per workgroup (pipeline fill and the
  // partial-state write) and the reduction of the partial states.
  StatePlan best{1, c->page_size, 1, std::max(n_pages, 1)};
  if (n_pages <= 0) return best;
  const long bh = (long)c->batch * c->num_heads;
  constexpr double kGroupTiles = 2.5, kReduceTilesPerGroup = 0.004;
  double best_cost = 1e300;
  for (int parts = 1; parts <= 16; ++parts) {
    int len = (c->page_size + parts - 1) / parts;
    len = (len + 7) / 8 * 8;
    const int parts_eff = (c->page_size + len - 1) / len;
    if (parts > 1 && parts_eff != parts) continue;  // same split as a smaller count
    // every unit must end at key >= 64 (the kernel's tile window)
    if (parts > 1 && c->page_size >= 64 && len < 64) break;
    const long units = (long)n_pages * parts_eff;
    const int tiles = (len + 63) / 64;
    for (int r = 1; r <= 8; ++r) {
      const long gpb = (long)r * kStateTargetGroups / bh;  // groups per (b, h)
      if (gpb < 1) continue;
      const long upw = (units + gpb - 1) / gpb;
      const long groups = (units + upw - 1) / upw;
      const long g_all = bh * groups;
      const long rounds = (g_all + kStateTargetGroups - 1) / kStateTargetGroups;
      const double cost = rounds * (upw * (double)tiles + kGroupTiles) + kReduceTilesPerGroup * g_all;
      if (cost < best_cost * 0.999) {
        best_cost = cost;
        best = StatePlan{parts_eff, len, (int)upw, (int)groups};
      }
    }
  }
  return best;
}

struct StateWs {
  size_t s_off, z_off, k_off, total;
};

StateWs state_ws(const hsa_config_t* c, int n_pages, const StatePlan& pl) {
  const size_t bh = (size_t)c->batch * c->num_heads, d = c->head_dim;
  StateWs w;
  w.s_off = 0;
  w.z_off = align_up(bh * pl.n_groups * d * d * 4);
  w.k_off = w.z_off + align_up(bh * pl.n_groups * d * 4);
  w.total = w.k_off + align_up(bh * (size_t)n_pages * pl.parts * d * 8);
  return w;
}

int qsum_splits(int n_q) { return (n_q + kQsumRows - 1) / kQsumRows; }

size_t select_ws_bytes(const hsa_config_t* c, int n_q) {
  return align_up((size_t)c->batch * qsum_splits(n_q) * c->num_heads * c->head_dim * 8);
}

size_t sel_ws_bytes(const hsa_config_t* c, int k_max) {
  return align_up((size_t)c->batch * c->num_heads * std::max(k_max, 1) * 4);
}

// partial outputs of split key lists (bf16 kernels only)
size_t partial_ws_bytes(const hsa_config_t* c, int n_q) {
  if (c->dtype != HSA_DTYPE_BF16) return 0;
  return attention_partial_bytes(c->batch, c->num_heads, c->head_dim, n_q, kPartPerHead * c->num_heads);
}

// Split partials of a planned launch: the schedule's p.sc.n_part slots (at
// most kPartPerHead * H, what partial_ws_bytes provides for), then the LSE
// partials, then the arrival counters of the split query tiles.
void set_partials(AttnParams& p, const hsa_config_t* c, int n_q, void* base) {
  uint8_t* b = static_cast<uint8_t*>(base);
  const size_t o_bytes = attention_partial_o_bytes(c->batch, c->head_dim, n_q, p.sc.n_part);
  p.part_o = reinterpret_cast<float*>(b);
  p.part_lse = reinterpret_cast<float*>(b + o_bytes);
  p.attn_ctr = reinterpret_cast<int32_t*>(b + o_bytes + attention_partial_lse_bytes(c->batch, n_q, p.sc.n_part));
}

// Bytes of split partials a planned launch writes.
size_t planned_partial_bytes(const AttnParams& p, const hsa_config_t* c, int n_q) {
  if (c->dtype != HSA_DTYPE_BF16 || p.sc.n_part == 0) return 0;
  return attention_partial_bytes(c->batch, c->num_heads, c->head_dim, n_q, p.sc.n_part);
}

hsa_status_t from_hip(hipError_t e) { return e == hipSuccess ? HSA_OK : HSA_ERR_DEVICE; }

hsa_status_t check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return HSA_OK;
  if (!ws || have < need) return HSA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return HSA_ERR_WORKSPACE;
  return HSA_OK;
}

hsa_status_t check_budgets(const hsa_config_t* c, const int32_t* k_h, int k_max) {
  if (k_max < 0) return HSA_ERR_INVALID_ARG;
  if (!k_h) return HSA_OK;
  for (int h = 0; h < c->num_heads; ++h)
    if (k_h[h] < 0 || k_h[h] > k_max) return HSA_ERR_INVALID_ARG;
  return HSA_OK;
}

// ---------------------------------------------------------------- block-sparse mode
static_assert(kQsumRows * 2 == kBlockQ, "query blocks are two query-sum splits");

int blocks_per_page(int P, int B) { return (P + B - 1) / B; }

int block_count(const hsa_config_t* c, int n_hist, int n_cur) {
  return n_hist * blocks_per_page(c->page_size, kBlockHist) +
         n_cur * blocks_per_page(c->page_size, kBlockCur);
}

// Workspace of the adaptive calls: [query sums][sel][block means][sorted
// rows: running weight, block id][Gini terms][tile lists][list lengths]
// [partial outputs].
struct AdaptiveWs {
  int n_qb, n_qt, n_blk_max, n_pad, cap, rpg;
  size_t sel_off, kbar_off, rc_off, ri_off, rg_off, bl_off, bll_off, part_off, total;
};

AdaptiveWs adaptive_ws(const hsa_config_t* c, int n_q, int k_max, int n_cur) {
  AdaptiveWs w{};
  const size_t bh = (size_t)c->batch * c->num_heads, d = c->head_dim;
  w.n_qb = (n_q + kBlockQ - 1) / kBlockQ;
  w.n_qt = (n_q + 2 * kBlockQ - 1) / (2 * kBlockQ);
  w.n_blk_max = block_count(c, k_max, n_cur);
  w.n_pad = 64;
  while (w.n_pad < w.n_blk_max) w.n_pad <<= 1;
  w.cap = std::max(1, (k_max + n_cur) * blocks_per_page(c->page_size, 64));
  w.rpg = 4;
  while (w.rpg > 1 && block_rows_lds_bytes(c->head_dim, w.n_pad, w.rpg) > 65536) w.rpg >>= 1;
  const size_t nb = std::max(1, w.n_blk_max);
  w.sel_off = select_ws_bytes(c, n_q);
  w.kbar_off = w.sel_off + sel_ws_bytes(c, k_max);
  w.rc_off = w.kbar_off + align_up(bh * d * nb * 8);
  w.ri_off = w.rc_off + align_up(bh * w.n_qb * nb * 8);
  w.rg_off = w.ri_off + align_up(bh * w.n_qb * nb * 4);
  w.bl_off = w.rg_off + align_up(bh * w.n_qb * 8);
  w.bll_off = w.bl_off + align_up(bh * w.n_qt * (size_t)w.cap * 8);
  w.part_off = w.bll_off + align_up(bh * w.n_qt * 4);
  w.total = w.part_off + partial_ws_bytes(c, n_q);
  return w;
}

hsa_status_t check_taus(double tau_min, double tau_max) {
  if (!(tau_min >= 0.0 && tau_min <= tau_max && tau_max <= 1.0)) return HSA_ERR_INVALID_ARG;
  return HSA_OK;
}

double pooled_scale(const hsa_config_t* c) {
  return c->sm_scale > 0.f ? (double)c->sm_scale : 1.0 / sqrt((double)c->head_dim);
}

// Outputs of the selection that hsa_block_select exposes (all nullable).
struct BlockSelOut {
  double* gini = nullptr;
  double* tau = nullptr;
  int32_t* n_kept = nullptr;
  int32_t* kept = nullptr;
  double* pooled = nullptr;
  int32_t kept_len = 0;
};

// Block selection over the lists of sel + [cur_first, cur_first + n_cur);
// the query sums are computed first unless the page selection already left
// them in the workspace.
hsa_status_t run_block_select(const hsa_config_t* c, const void* q, int n_q,
                              const hsa_kv_pool_t* pool, const int32_t* sel, int k_max,
                              int cur_first, int n_cur, double tau_min, double tau_max,
                              const AdaptiveWs& w, uint8_t* base, bool have_qsum,
                              const BlockSelOut& out, hipStream_t s) {
  QsumParams qp{};
  qp.q = q;
  qp.n_q = n_q;
  qp.HD = c->num_heads * c->head_dim;
  qp.rows_per_split = kQsumRows;
  qp.n_split = qsum_splits(n_q);
  qp.ws_qs = reinterpret_cast<double*>(base);
  if (!have_qsum) {
    const hipError_t e = launch_qsum(c->dtype, c->batch, qp, s);
    if (e != hipSuccess) return HSA_ERR_DEVICE;
  }
  BlockSelParams p{};
  p.k = pool->k;
  p.page_table = pool->page_table;
  p.sel = sel;
  p.H = c->num_heads;
  p.P = c->page_size;
  p.n_q = n_q;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.k_max = k_max;
  p.cur_first = cur_first;
  p.n_cur = n_cur;
  p.n_qb = w.n_qb;
  p.n_qt = w.n_qt;
  p.n_blk_max = w.n_blk_max;
  p.n_pad = w.n_pad;
  p.rpg = w.rpg;
  p.qs_split = qp.n_split;
  p.scale = pooled_scale(c);
  p.tau_min = tau_min;
  p.tau_max = tau_max;
  p.ws_qs = qp.ws_qs;
  p.kbar_t = reinterpret_cast<double*>(base + w.kbar_off);
  p.row_c = reinterpret_cast<double*>(base + w.rc_off);
  p.row_i = reinterpret_cast<int32_t*>(base + w.ri_off);
  p.row_g = reinterpret_cast<double*>(base + w.rg_off);
  p.blist = reinterpret_cast<int2*>(base + w.bl_off);
  p.blist_len = reinterpret_cast<int32_t*>(base + w.bll_off);
  p.blist_cap = w.cap;
  p.gini = out.gini;
  p.tau = out.tau;
  p.n_kept = out.n_kept;
  p.kept = out.kept;
  p.kept_len = out.kept_len;
  p.pooled = out.pooled;
  return from_hip(launch_block_select(c->dtype, c->head_dim, c->batch, p, s));
}

void set_block_lists(AttnParams& p, const AdaptiveWs& w, uint8_t* base) {
  p.blist = reinterpret_cast<const int2*>(base + w.bl_off);
  p.blist_len = reinterpret_cast<const int32_t*>(base + w.bll_off);
  p.blist_cap = w.cap;
}

// Checks shared by the adaptive calls on top of their base call's checks.
hsa_status_t check_adaptive(const hsa_config_t* c, int n_q, int k_max, int n_cur, double tau_min,
                            double tau_max) {
  hsa_status_t st = check_taus(tau_min, tau_max);
  if (st != HSA_OK) return st;
  if (block_count(c, k_max, n_cur) > HSA_MAX_BLOCKS) return HSA_ERR_UNSUPPORTED;
  (void)n_q;
  return HSA_OK;
}

// ---------------------------------------------------------------- Linformer branch
bool valid_rank(int r) { return r == 32 || r == 64 || r == 128; }

struct CompressPlan {
  int parts, part_len;
};

// A page is split into parts (each a multiple of 64 tokens) only when there
// are too few (page, head) pairs to give every CU a workgroup; parts add an
// fp32 partial write and a reduction (64 KB per part at rank 64, d = 128).
CompressPlan plan_compress(const hsa_config_t* c, int n_pages) {
  const int tiles = (c->page_size + 63) / 64;
  const long items = (long)c->batch * c->num_heads * std::max(n_pages, 1);
  int parts = 1;
  if (c->dtype == HSA_DTYPE_BF16 && items < 256) parts = (int)std::min<long>(tiles, (256 + items - 1) / items);
  const int part_len = (tiles + parts - 1) / parts * 64;
  return CompressPlan{(c->page_size + part_len - 1) / part_len, part_len};
}

size_t compress_ws_bytes(const hsa_config_t* c, int rank, int n_pages, const CompressPlan& pl) {
  if (pl.parts <= 1) return 0;
  return align_up((size_t)c->batch * c->num_heads * n_pages * pl.parts * 2 * rank * c->head_dim * 4);
}

size_t o_lin_bytes(const hsa_config_t* c, int n_q) {
  return align_up((size_t)c->batch * n_q * c->num_heads * c->head_dim * 4);
}

hsa_status_t run_select(const hsa_config_t* c, const void* q, int n_q, const double* kmean,
                        int max_pages, int n_cand, const int32_t* k_h, int k_max, int32_t* sel,
                        double* sel_score, void* ws, hipStream_t s,
                        const int32_t* cand_range = nullptr) {
  QsumParams qp{};
  qp.q = q;
  qp.n_q = n_q;
  qp.HD = c->num_heads * c->head_dim;
  qp.rows_per_split = kQsumRows;
  qp.n_split = qsum_splits(n_q);
  qp.ws_qs = static_cast<double*>(ws);
  SelectParams sp{};
  sp.ws_qs = qp.ws_qs;
  sp.page_kmean = kmean;
  sp.H = c->num_heads;
  sp.n_q = n_q;
  sp.n_split = qp.n_split;
  sp.max_pages = max_pages;
  sp.n_cand = n_cand;
  sp.k_max = k_max;
  for (int h = 0; h < c->num_heads; ++h) sp.k_h[h] = k_h[h];
  sp.sel = sel;
  sp.sel_score = sel_score;
  sp.cand_range = cand_range;
  return from_hip(launch_page_select(c->dtype, c->head_dim, c->batch, qp, sp, s));
}

hsa_status_t check_sparse(const hsa_config_t* cfg, const void* q, int32_t n_q,
                          const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                          const int32_t* k_h, int32_t cur_first_page, int32_t n_cur_pages,
                          const float* o_sp) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!q || !o_sp || n_q < 1 || k_max < 0 || n_cur_pages < 0 || cur_first_page < 0)
    return HSA_ERR_INVALID_ARG;
  if (k_max > 0 && !sel) return HSA_ERR_INVALID_ARG;
  if (k_max == 0 && n_cur_pages == 0) return HSA_ERR_INVALID_ARG;
  if ((long)cur_first_page + n_cur_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if ((long)k_max + n_cur_pages > HSA_MAX_LIST) return HSA_ERR_UNSUPPORTED;
  return check_budgets(cfg, k_h, k_max);
}

// The sparse branch alone; w != NULL walks the tile lists of a block
// selection already in the workspace.
hsa_status_t run_sparse(const hsa_config_t* cfg, const void* q, int32_t n_q,
                        const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                        const int32_t* k_h, int32_t cur_first_page, int32_t n_cur_pages,
                        float* o_sp, float* lse, void* partials, const AdaptiveWs* w,
                        hipStream_t s) {
  AttnParams p{};
  p.q = q;
  p.k = pool->k;
  p.v = pool->v;
  p.page_table = pool->page_table;
  p.sel = sel;  // not read when k_max == 0
  p.H = cfg->num_heads;
  p.P = cfg->page_size;
  p.n_q = n_q;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.k_max = k_max;
  p.cur_first = cur_first_page;
  p.n_cur = n_cur_pages;
  p.sm_scale = softmax_scale(cfg);
  p.scale_log2 = p.sm_scale * 1.4426950408889634f;
  p.mode = ATTN_SPARSE;
  p.o_sp = o_sp;
  p.lse = lse;
  int list_len[HSA_MAX_HEADS];
  for (int h = 0; h < cfg->num_heads; ++h)
    list_len[h] = std::min(k_h ? k_h[h] : k_max, pool->max_pages) + n_cur_pages;
  if (!plan_attention(p, cfg->batch, cfg->num_heads, cfg->head_dim, n_q, cfg->page_size, list_len,
                      kPartPerHead * cfg->num_heads, cfg->dtype == HSA_DTYPE_BF16, w ? 4 : kPageWaves))
    return HSA_ERR_UNSUPPORTED;
  if (cfg->dtype == HSA_DTYPE_BF16) set_partials(p, cfg, n_q, partials);
  if (w) set_block_lists(p, *w, static_cast<uint8_t*>(partials) - w->part_off);
  return from_hip(launch_attention(cfg->dtype, cfg->head_dim, cfg->batch, p, s));
}

}  // namespace

extern "C" {

const char* hsa_status_string(hsa_status_t s) {
  switch (s) {
    case HSA_OK: return "HSA_OK";
    case HSA_ERR_INVALID_ARG: return "HSA_ERR_INVALID_ARG";
    case HSA_ERR_UNSUPPORTED: return "HSA_ERR_UNSUPPORTED";
    case HSA_ERR_OUT_OF_RANGE: return "HSA_ERR_OUT_OF_RANGE";
    case HSA_ERR_WORKSPACE: return "HSA_ERR_WORKSPACE";
    case HSA_ERR_DEVICE: return "HSA_ERR_DEVICE";
    case HSA_ERR_IO: return "HSA_ERR_IO";
  }
  return "HSA_ERR_UNKNOWN";
}

size_t hsa_state_update_workspace_size(const hsa_config_t* cfg, int32_t n_pages) {
  if (check_cfg(cfg) != HSA_OK || n_pages < 0) return 0;
  if (n_pages == 0) return 0;
  return state_ws(cfg, n_pages, plan_state(cfg, n_pages)).total;
}

size_t hsa_page_select_workspace_size(const hsa_config_t* cfg, int32_t n_q) {
  if (check_cfg(cfg) != HSA_OK || n_q < 1) return 0;
  return select_ws_bytes(cfg, n_q);
}

size_t hsa_sparse_attn_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                      int32_t n_cur_pages) {
  if (check_cfg(cfg) != HSA_OK || n_q < 1 || k_max < 0 || n_cur_pages < 0) return 0;
  return partial_ws_bytes(cfg, n_q);
}

size_t hsa_forward_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                  int32_t n_cur_pages) {
  if (check_cfg(cfg) != HSA_OK || n_q < 1 || k_max < 0 || n_cur_pages < 0) return 0;
  return select_ws_bytes(cfg, n_q) + sel_ws_bytes(cfg, k_max) + partial_ws_bytes(cfg, n_q);
}

hsa_status_t hsa_state_update(const hsa_config_t* cfg, const hsa_kv_pool_t* pool,
                              int32_t first_page, int32_t n_pages, float* kv_state,
                              float* k_state, double* page_kmean, void* ws, size_t ws_bytes,
                              void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!kv_state || !k_state || !page_kmean) return HSA_ERR_INVALID_ARG;
  if (first_page < 0 || n_pages < 0) return HSA_ERR_INVALID_ARG;
  if ((long)first_page + n_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if (n_pages == 0) return HSA_OK;
  const StatePlan pl = plan_state(cfg, n_pages);
  const StateWs w = state_ws(cfg, n_pages, pl);
  if ((st = check_ws(ws, ws_bytes, w.total)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, first_page, n_pages, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  StateParams p{};
  p.k = pool->k;
  p.v = pool->v;
  p.page_table = pool->page_table;
  p.H = cfg->num_heads;
  p.P = cfg->page_size;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.first_page = first_page;
  p.n_pages = n_pages;
  p.parts = pl.parts;
  p.part_len = pl.part_len;
  p.upw = pl.upw;
  p.n_groups = pl.n_groups;
  p.ws_S = reinterpret_cast<float*>(base + w.s_off);
  p.ws_z = reinterpret_cast<float*>(base + w.z_off);
  p.ws_k = reinterpret_cast<double*>(base + w.k_off);
  StateReduceParams r{};
  r.kv_state = kv_state;
  r.k_state = k_state;
  r.page_kmean = page_kmean;
  r.ws_S = p.ws_S;
  r.ws_z = p.ws_z;
  r.ws_k = p.ws_k;
  r.H = cfg->num_heads;
  r.P = cfg->page_size;
  r.max_pages = pool->max_pages;
  r.first_page = first_page;
  r.n_pages = n_pages;
  r.parts = pl.parts;
  r.n_groups = pl.n_groups;
  return from_hip(launch_state_update(cfg->dtype, cfg->head_dim, cfg->batch, p, r, s));
}

hsa_status_t hsa_page_write(const hsa_config_t* cfg, const hsa_kv_pool_t* pool, const void* k_src,
                            const void* v_src, int32_t first_page, int32_t n_pages,
                            const int32_t* src_of, void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!k_src || !v_src || first_page < 0 || n_pages < 0) return HSA_ERR_INVALID_ARG;
  if ((long)first_page + n_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if (n_pages == 0) return HSA_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, first_page, n_pages, s)) != HSA_OK) return st;
  PageWriteParams p{};
  // the pool is the caller's device memory; this call is the one that writes it
  p.k = const_cast<void*>(pool->k);
  p.v = const_cast<void*>(pool->v);
  p.page_table = pool->page_table;
  p.k_src = k_src;
  p.v_src = v_src;
  p.src_of = src_of;
  p.H = cfg->num_heads;
  p.P = cfg->page_size;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.first_page = first_page;
  p.n_pages = n_pages;
  return from_hip(launch_page_write(cfg->dtype, cfg->head_dim, cfg->batch, p, s));
}

int32_t hsa_cube_order(int32_t frames, int32_t height, int32_t width, int32_t ct, int32_t ch,
                       int32_t cw, int32_t* src_of) {
  if (frames < 1 || height < 1 || width < 1 || ct < 1 || ch < 1 || cw < 1 || !src_of) return -1;
  if ((long)frames * height * width > (1L << 30)) return -1;
  return cube_order(frames, height, width, ct, ch, cw, src_of);
}

hsa_status_t hsa_page_select(const hsa_config_t* cfg, const void* q, int32_t n_q,
                             const double* page_kmean, int32_t max_pages, int32_t n_cand,
                             const int32_t* k_h, int32_t k_max, int32_t* sel, double* sel_score,
                             void* ws, size_t ws_bytes, void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if (!q || !page_kmean || !k_h || !sel) return HSA_ERR_INVALID_ARG;
  if (n_q < 1 || n_cand < 0 || max_pages < 1 || k_max < 1) return HSA_ERR_INVALID_ARG;
  if (n_cand > max_pages) return HSA_ERR_OUT_OF_RANGE;
  if (n_cand > HSA_MAX_CAND) return HSA_ERR_UNSUPPORTED;
  if ((st = check_budgets(cfg, k_h, k_max)) != HSA_OK) return st;
  if ((st = check_ws(ws, ws_bytes, select_ws_bytes(cfg, n_q))) != HSA_OK) return st;
  return run_select(cfg, q, n_q, page_kmean, max_pages, n_cand, k_h, k_max, sel, sel_score, ws,
                    static_cast<hipStream_t>(stream));
}

hsa_status_t hsa_sparse_attn(const hsa_config_t* cfg, const void* q, int32_t n_q,
                             const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                             const int32_t* k_h, int32_t cur_first_page, int32_t n_cur_pages,
                             float* o_sp, float* lse, void* ws, size_t ws_bytes, void* stream) {
  hsa_status_t st = check_sparse(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages,
                                 o_sp);
  if (st != HSA_OK) return st;
  if ((st = check_ws(ws, ws_bytes, partial_ws_bytes(cfg, n_q))) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, cur_first_page, n_cur_pages, s)) != HSA_OK) return st;
  if ((st = validate_selection(cfg, pool, sel, k_max, s)) != HSA_OK) return st;
  return run_sparse(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages, o_sp, lse, ws,
                    nullptr, s);
}

size_t hsa_adaptive_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                   int32_t n_cur_pages) {
  if (check_cfg(cfg) != HSA_OK || n_q < 1 || k_max < 0 || n_cur_pages < 0) return 0;
  if ((long)k_max + n_cur_pages > HSA_MAX_LIST) return 0;
  return adaptive_ws(cfg, n_q, k_max, n_cur_pages).total;
}

hsa_status_t hsa_attention_plan(const hsa_config_t* cfg, int32_t n_q, const int32_t* list_len,
                                int32_t adaptive, int32_t* n_items, int32_t* n_chunks,
                                int32_t* max_split) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if (!list_len || n_q < 1) return HSA_ERR_INVALID_ARG;
  for (int h = 0; h < cfg->num_heads; ++h)
    if (list_len[h] < 1 || list_len[h] > HSA_MAX_LIST) return HSA_ERR_INVALID_ARG;
  AttnParams p{};
  if (!plan_attention(p, cfg->batch, cfg->num_heads, cfg->head_dim, n_q, cfg->page_size, list_len,
                      kPartPerHead * cfg->num_heads, cfg->dtype == HSA_DTYPE_BF16,
                      adaptive ? 4 : kPageWaves))
    return HSA_ERR_UNSUPPORTED;
  int widest = 1;
  for (int h = 0; h < cfg->num_heads; ++h) widest = std::max(widest, (int)p.sc.n_split[h]);
  if (n_items) *n_items = p.sc.n_items;
  if (n_chunks) *n_chunks = p.sc.n_chunks;
  if (max_split) *max_split = widest;
  return HSA_OK;
}

int32_t hsa_block_count(const hsa_config_t* cfg, int32_t n_hist_pages, int32_t n_cur_pages) {
  if (check_cfg(cfg) != HSA_OK || n_hist_pages < 0 || n_cur_pages < 0) return -1;
  if ((long)n_hist_pages + n_cur_pages > HSA_MAX_LIST) return -1;
  return block_count(cfg, n_hist_pages, n_cur_pages);
}

hsa_status_t hsa_block_select(const hsa_config_t* cfg, const void* q, int32_t n_q,
                              const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                              int32_t cur_first_page, int32_t n_cur_pages, double tau_min,
                              double tau_max, double* gini, double* tau, int32_t* n_kept,
                              int32_t* kept, double* pooled, int32_t kept_len, void* ws,
                              size_t ws_bytes, void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!q || n_q < 1 || k_max < 0 || n_cur_pages < 0 || cur_first_page < 0)
    return HSA_ERR_INVALID_ARG;
  if (k_max > 0 && !sel) return HSA_ERR_INVALID_ARG;
  if (k_max == 0 && n_cur_pages == 0) return HSA_ERR_INVALID_ARG;
  if ((long)cur_first_page + n_cur_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if ((long)k_max + n_cur_pages > HSA_MAX_LIST) return HSA_ERR_UNSUPPORTED;
  if ((st = check_adaptive(cfg, n_q, k_max, n_cur_pages, tau_min, tau_max)) != HSA_OK) return st;
  if ((kept || pooled) && kept_len < block_count(cfg, k_max, n_cur_pages)) return HSA_ERR_INVALID_ARG;
  const AdaptiveWs w = adaptive_ws(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, w.total)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, cur_first_page, n_cur_pages, s)) != HSA_OK) return st;
  if ((st = validate_selection(cfg, pool, sel, k_max, s)) != HSA_OK) return st;
  BlockSelOut out;
  out.gini = gini;
  out.tau = tau;
  out.n_kept = n_kept;
  out.kept = kept;
  out.pooled = pooled;
  out.kept_len = kept_len;
  return run_block_select(cfg, q, n_q, pool, sel, k_max, cur_first_page, n_cur_pages, tau_min,
                          tau_max, w, static_cast<uint8_t*>(ws), false, out, s);
}

hsa_status_t hsa_sparse_attn_adaptive(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                      const hsa_kv_pool_t* pool, const int32_t* sel,
                                      int32_t k_max, const int32_t* k_h, int32_t cur_first_page,
                                      int32_t n_cur_pages, double tau_min, double tau_max,
                                      float* o_sp, float* lse, void* ws, size_t ws_bytes,
                                      void* stream) {
  hsa_status_t st = check_sparse(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages,
                                 o_sp);
  if (st != HSA_OK) return st;
  if ((st = check_adaptive(cfg, n_q, k_max, n_cur_pages, tau_min, tau_max)) != HSA_OK) return st;
  const AdaptiveWs w = adaptive_ws(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, w.total)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, cur_first_page, n_cur_pages, s)) != HSA_OK) return st;
  if ((st = validate_selection(cfg, pool, sel, k_max, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  st = run_block_select(cfg, q, n_q, pool, sel, k_max, cur_first_page, n_cur_pages, tau_min,
                        tau_max, w, base, false, BlockSelOut(), s);
  if (st != HSA_OK) return st;
  return run_sparse(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages, o_sp, lse,
                    base + w.part_off, &w, s);
}

}  // extern "C"

namespace {

// Checks shared by hsa_forward and hsa_forward_selected.
// need_state: the kernelised linear branch reads kv_state / k_state.
hsa_status_t check_forward(const hsa_config_t* cfg, const void* q, int32_t n_q,
                           const hsa_kv_pool_t* pool, int32_t n_cand, int32_t n_cur_pages,
                           const int32_t* k_h, int32_t k_max, const float* kv_state,
                           const float* k_state, const void* o, bool need_state = true) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!q || !k_h || !o) return HSA_ERR_INVALID_ARG;
  if (need_state && (!kv_state || !k_state)) return HSA_ERR_INVALID_ARG;
  if (n_q < 1 || n_cand < 0 || n_cur_pages < 0 || k_max < 1) return HSA_ERR_INVALID_ARG;
  if ((long)n_cand + n_cur_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if (n_cand > HSA_MAX_CAND) return HSA_ERR_UNSUPPORTED;
  if ((long)k_max + n_cur_pages > HSA_MAX_LIST) return HSA_ERR_UNSUPPORTED;
  if ((st = check_budgets(cfg, k_h, k_max)) != HSA_OK) return st;
  for (int h = 0; h < cfg->num_heads; ++h)
    if (n_cur_pages == 0 && std::min(k_h[h], n_cand) == 0) return HSA_ERR_INVALID_ARG;
  return HSA_OK;
}

// Schedule of the attention launch of the forward calls: each head's list
// is its selected pages (at most n_cand) plus the current pages.
bool plan_attend(AttnParams& p, const hsa_config_t* cfg, int n_q, const int32_t* k_h, int n_cand,
                 int n_cur_pages, bool tile_lists) {
  int list_len[HSA_MAX_HEADS];
  for (int h = 0; h < cfg->num_heads; ++h) list_len[h] = std::min(k_h[h], n_cand) + n_cur_pages;
  return plan_attention(p, cfg->batch, cfg->num_heads, cfg->head_dim, n_q, cfg->page_size, list_len,
                        kPartPerHead * cfg->num_heads, cfg->dtype == HSA_DTYPE_BF16,
                        tile_lists ? 4 : kPageWaves);
}

// Sparse branch + linear branch + gated fusion for a selection in `sel`.
hsa_status_t run_attend(const hsa_config_t* cfg, const void* q, int32_t n_q,
                        const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                        const int32_t* k_h, int32_t n_cand, int32_t n_cur_pages,
                        const float* kv_state, const float* k_state, const float* g_lin,
                        const float* g_sp, void* o, void* partials, hipStream_t s,
                        const AdaptiveWs* w = nullptr, uint8_t* wbase = nullptr,
                        const float* o_lin = nullptr) {
  AttnParams p{};
  p.o_lin = o_lin;
  p.q = q;
  p.k = pool->k;
  p.v = pool->v;
  p.page_table = pool->page_table;
  p.sel = sel;
  p.H = cfg->num_heads;
  p.P = cfg->page_size;
  p.n_q = n_q;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.k_max = k_max;
  p.cur_first = n_cand;
  p.n_cur = n_cur_pages;
  p.sm_scale = softmax_scale(cfg);
  p.scale_log2 = p.sm_scale * 1.4426950408889634f;
  p.mode = ATTN_FINAL;
  p.kv_state = kv_state;
  p.k_state = k_state;
  p.g_lin = g_lin;
  p.g_sp = g_sp;
  p.gate_elem = cfg->gate_dims > 1;
  p.o = o;
  if (!plan_attend(p, cfg, n_q, k_h, n_cand, n_cur_pages, w != nullptr)) return HSA_ERR_UNSUPPORTED;
  if (cfg->dtype == HSA_DTYPE_BF16) set_partials(p, cfg, n_q, partials);
  if (w) set_block_lists(p, *w, wbase);
  return from_hip(launch_attention(cfg->dtype, cfg->head_dim, cfg->batch, p, s));
}

// hsa_forward after its checks: page selection into sel_out (or the
// workspace), then the attention launch. Workspace layout: [query sums]
// [selection][split partials].
hsa_status_t forward_body(const hsa_config_t* cfg, const void* q, int32_t n_q,
                          const hsa_kv_pool_t* pool, int32_t n_cand, int32_t n_cur_pages,
                          const int32_t* k_h, int32_t k_max, const float* kv_state,
                          const float* k_state, const double* page_kmean, const float* g_lin,
                          const float* g_sp, void* o, int32_t* sel_out, uint8_t* base,
                          hipStream_t s) {
  int32_t* sel = sel_out ? sel_out : reinterpret_cast<int32_t*>(base + select_ws_bytes(cfg, n_q));
  void* partials = base + select_ws_bytes(cfg, n_q) + sel_ws_bytes(cfg, k_max);
  hsa_status_t st =
      run_select(cfg, q, n_q, page_kmean, pool->max_pages, n_cand, k_h, k_max, sel, nullptr, base, s);
  if (st != HSA_OK) return st;
  return run_attend(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, kv_state, k_state,
                    g_lin, g_sp, o, partials, s);
}

}  // namespace

extern "C" {

hsa_status_t hsa_forward(const hsa_config_t* cfg, const void* q, int32_t n_q,
                         const hsa_kv_pool_t* pool, int32_t n_cand, int32_t n_cur_pages,
                         const int32_t* k_h, int32_t k_max, const float* kv_state,
                         const float* k_state, const double* page_kmean, const float* g_lin,
                         const float* g_sp, void* o, int32_t* sel_out, void* ws, size_t ws_bytes,
                         void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state,
                                  k_state, o);
  if (st != HSA_OK) return st;
  if (!page_kmean) return HSA_ERR_INVALID_ARG;
  const size_t need = hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, need)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, 0, n_cand + n_cur_pages, s)) != HSA_OK) return st;
  return forward_body(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                      page_kmean, g_lin, g_sp, o, sel_out, static_cast<uint8_t*>(ws), s);
}

hsa_status_t hsa_forward_selected(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                  const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                                  const int32_t* k_h, int32_t n_cand, int32_t n_cur_pages,
                                  const float* kv_state, const float* k_state,
                                  const float* g_lin, const float* g_sp, void* o, void* ws,
                                  size_t ws_bytes, void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state,
                                  k_state, o);
  if (st != HSA_OK) return st;
  if (!sel) return HSA_ERR_INVALID_ARG;
  const size_t need = hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, need)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, n_cand, n_cur_pages, s)) != HSA_OK) return st;
  if ((st = validate_selection(cfg, pool, sel, k_max, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  void* partials = base + select_ws_bytes(cfg, n_q) + sel_ws_bytes(cfg, k_max);
  return run_attend(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, kv_state, k_state,
                    g_lin, g_sp, o, partials, s);
}

hsa_status_t hsa_forward_adaptive(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                  const hsa_kv_pool_t* pool, int32_t n_cand,
                                  int32_t n_cur_pages, const int32_t* k_h, int32_t k_max,
                                  double tau_min, double tau_max, const float* kv_state,
                                  const float* k_state, const double* page_kmean,
                                  const float* g_lin, const float* g_sp, void* o,
                                  int32_t* sel_out, void* ws, size_t ws_bytes, void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state,
                                  k_state, o);
  if (st != HSA_OK) return st;
  if (!page_kmean) return HSA_ERR_INVALID_ARG;
  if ((st = check_adaptive(cfg, n_q, k_max, n_cur_pages, tau_min, tau_max)) != HSA_OK) return st;
  const AdaptiveWs w = adaptive_ws(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, w.total)) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, 0, n_cand + n_cur_pages, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  int32_t* sel = sel_out ? sel_out : reinterpret_cast<int32_t*>(base + w.sel_off);
  st = run_select(cfg, q, n_q, page_kmean, pool->max_pages, n_cand, k_h, k_max, sel, nullptr, ws, s);
  if (st != HSA_OK) return st;
  st = run_block_select(cfg, q, n_q, pool, sel, k_max, n_cand, n_cur_pages, tau_min, tau_max, w,
                        base, true, BlockSelOut(), s);
  if (st != HSA_OK) return st;
  return run_attend(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, kv_state, k_state,
                    g_lin, g_sp, o, base + w.part_off, s, &w, base);
}

hsa_status_t hsa_chunk_select(const hsa_config_t* cfg, const float* prompt_emb,
                              const float* chunk_emb, int32_t emb_dim, int32_t n_chunks,
                              const int32_t* chunk_first, int32_t n_cand, int32_t* chunk_out,
                              double* chunk_score, int32_t* cand_range, void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if (!prompt_emb || !chunk_emb || !chunk_first || !cand_range) return HSA_ERR_INVALID_ARG;
  if (emb_dim < 1 || n_chunks < 1 || n_cand < 0) return HSA_ERR_INVALID_ARG;
  ChunkSelectParams p{};
  p.prompt = prompt_emb;
  p.chunks = chunk_emb;
  p.chunk_first = chunk_first;
  p.E = emb_dim;
  p.M = n_chunks;
  p.n_cand = n_cand;
  p.chunk_out = chunk_out;
  p.chunk_score = chunk_score;
  p.cand_range = cand_range;
  return from_hip(launch_chunk_select(cfg->batch, p, static_cast<hipStream_t>(stream)));
}

size_t hsa_retrieval_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                    int32_t n_cur_pages) {
  const size_t f = hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages);
  return f ? f + align_up((size_t)cfg->batch * 2 * 4) : 0;
}

hsa_status_t hsa_forward_retrieval(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                   const hsa_kv_pool_t* pool, const float* prompt_emb,
                                   const float* chunk_emb, int32_t emb_dim, int32_t n_chunks,
                                   const int32_t* chunk_first, int32_t n_cand,
                                   int32_t n_cur_pages, const int32_t* k_h, int32_t k_max,
                                   const float* kv_state, const float* k_state,
                                   const double* page_kmean, const float* g_lin,
                                   const float* g_sp, void* o, int32_t* chunk_out,
                                   int32_t* sel_out, void* ws, size_t ws_bytes, void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state,
                                  k_state, o);
  if (st != HSA_OK) return st;
  if (!page_kmean || !prompt_emb || !chunk_emb || !chunk_first) return HSA_ERR_INVALID_ARG;
  if (emb_dim < 1 || n_chunks < 1) return HSA_ERR_INVALID_ARG;
  const size_t fwd = hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, fwd + align_up((size_t)cfg->batch * 2 * 4))) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, 0, n_cand + n_cur_pages, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  int32_t* range = reinterpret_cast<int32_t*>(base + fwd);
  st = hsa_chunk_select(cfg, prompt_emb, chunk_emb, emb_dim, n_chunks, chunk_first, n_cand,
                        chunk_out, nullptr, range, stream);
  if (st != HSA_OK) return st;
  int32_t* sel = sel_out ? sel_out : reinterpret_cast<int32_t*>(base + select_ws_bytes(cfg, n_q));
  void* partials = base + select_ws_bytes(cfg, n_q) + sel_ws_bytes(cfg, k_max);
  st = run_select(cfg, q, n_q, page_kmean, pool->max_pages, n_cand, k_h, k_max, sel, nullptr, ws, s,
                  range);
  if (st != HSA_OK) return st;
  return run_attend(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, kv_state, k_state,
                    g_lin, g_sp, o, partials, s);
}

size_t hsa_linformer_compress_workspace_size(const hsa_config_t* cfg, int32_t rank,
                                             int32_t n_pages) {
  if (check_cfg(cfg) != HSA_OK || !valid_rank(rank) || n_pages < 0) return 0;
  return compress_ws_bytes(cfg, rank, n_pages, plan_compress(cfg, n_pages));
}

hsa_status_t hsa_linformer_compress(const hsa_config_t* cfg, const hsa_kv_pool_t* pool,
                                    const void* e_k, const void* e_v, int32_t rank,
                                    int32_t first_page, int32_t n_pages, void* ck, void* cv,
                                    void* ws, size_t ws_bytes, void* stream) {
  hsa_status_t st = check_cfg(cfg);
  if (st != HSA_OK) return st;
  if ((st = check_pool(pool)) != HSA_OK) return st;
  if (!e_k || !e_v || !ck || !cv) return HSA_ERR_INVALID_ARG;
  if (!valid_rank(rank)) return HSA_ERR_UNSUPPORTED;
  if (first_page < 0 || n_pages < 0) return HSA_ERR_INVALID_ARG;
  if ((long)first_page + n_pages > pool->max_pages) return HSA_ERR_OUT_OF_RANGE;
  if (n_pages == 0) return HSA_OK;
  const CompressPlan pl = plan_compress(cfg, n_pages);
  if ((st = check_ws(ws, ws_bytes, compress_ws_bytes(cfg, rank, n_pages, pl))) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, first_page, n_pages, s)) != HSA_OK) return st;
  CompressParams p{};
  p.k = pool->k;
  p.v = pool->v;
  p.page_table = pool->page_table;
  p.e_k = e_k;
  p.e_v = e_v;
  p.ck = ck;
  p.cv = cv;
  p.partial = static_cast<float*>(ws);
  p.H = cfg->num_heads;
  p.P = cfg->page_size;
  p.R = rank;
  p.D = cfg->head_dim;
  p.num_slots = pool->num_slots;
  p.max_pages = pool->max_pages;
  p.first_page = first_page;
  p.n_pages = n_pages;
  p.parts = pl.parts;
  p.part_len = pl.part_len;
  return from_hip(launch_compress(cfg->dtype, cfg->batch, p, s));
}

size_t hsa_linformer_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                    int32_t n_cur_pages) {
  const size_t a = hsa_adaptive_workspace_size(cfg, n_q, k_max, n_cur_pages);
  return a ? a + o_lin_bytes(cfg, n_q) : 0;
}

hsa_status_t hsa_forward_linformer(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                   const hsa_kv_pool_t* pool, const void* ck, const void* cv,
                                   int32_t rank, int32_t n_cand, int32_t n_cur_pages,
                                   const int32_t* k_h, int32_t k_max, double tau_min,
                                   double tau_max, const double* page_kmean, const float* g_lin,
                                   const float* g_sp, void* o, int32_t* sel_out, void* ws,
                                   size_t ws_bytes, void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, nullptr,
                                  nullptr, o, false);
  if (st != HSA_OK) return st;
  if (!page_kmean || !ck || !cv) return HSA_ERR_INVALID_ARG;
  if (!valid_rank(rank)) return HSA_ERR_UNSUPPORTED;
  if ((st = check_adaptive(cfg, n_q, k_max, n_cur_pages, tau_min, tau_max)) != HSA_OK) return st;
  const AdaptiveWs w = adaptive_ws(cfg, n_q, k_max, n_cur_pages);
  if ((st = check_ws(ws, ws_bytes, w.total + o_lin_bytes(cfg, n_q))) != HSA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, 0, n_cand + n_cur_pages, s)) != HSA_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(ws);
  float* o_lin = reinterpret_cast<float*>(base + w.total);
  int32_t* sel = sel_out ? sel_out : reinterpret_cast<int32_t*>(base + w.sel_off);
  st = run_select(cfg, q, n_q, page_kmean, pool->max_pages, n_cand, k_h, k_max, sel, nullptr, ws, s);
  if (st != HSA_OK) return st;
  st = run_block_select(cfg, q, n_q, pool, sel, k_max, n_cand, n_cur_pages, tau_min, tau_max, w,
                        base, true, BlockSelOut(), s);
  if (st != HSA_OK) return st;
  // linear branch: attention over the compressed pages of the same list (a
  // pool of page size rank through the same page table)
  hsa_config_t cr = *cfg;
  cr.page_size = rank;
  const hsa_kv_pool_t cpool{ck, cv, pool->page_table, pool->num_slots, pool->max_pages};
  st = run_sparse(&cr, q, n_q, &cpool, sel, k_max, k_h, n_cand, n_cur_pages, o_lin, nullptr,
                  base + w.part_off, nullptr, s);
  if (st != HSA_OK) return st;
  return run_attend(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, nullptr, nullptr,
                    g_lin, g_sp, o, base + w.part_off, s, &w, base, o_lin);
}

}  // extern "C"

// ---------------------------------------------------------------- no-allocation forward
// hsa_forward_noalloc runs hsa_forward with its workspace in `scratch`, a
// file-scope device array. Each GPU the library runs on holds its own copy
// (allocated when the code object is loaded on that device, kept until the
// process ends). In host code `scratch` names a host-side stand-in, not the
// device memory: its device address is taken once per device with
// hipGetSymbolAddress and only that address is ever passed to kernels.
// The forward kernels write every workspace byte they read within a call
// (query sums, selection, split partials), so nothing needs clearing.
namespace {

__device__ __align__(256) uint8_t scratch[HSA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (NULL on failure).
uint8_t* scratch_for_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = static_cast<uint8_t*>(ptr);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

size_t hsa_forward_noalloc_bytes(const hsa_config_t* cfg, int32_t n_q, int32_t n_cand,
                                 int32_t n_cur_pages, const int32_t* k_h, int32_t k_max) {
  if (check_cfg(cfg) != HSA_OK || !k_h || n_q < 1 || n_cand < 0 || n_cur_pages < 0 || k_max < 1)
    return 0;
  if (check_budgets(cfg, k_h, k_max) != HSA_OK) return 0;
  AttnParams p{};
  if (!plan_attend(p, cfg, n_q, k_h, n_cand, n_cur_pages, false)) return 0;
  return select_ws_bytes(cfg, n_q) + sel_ws_bytes(cfg, k_max) + planned_partial_bytes(p, cfg, n_q);
}

hsa_status_t hsa_forward_noalloc(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                 const hsa_kv_pool_t* pool, int32_t n_cand, int32_t n_cur_pages,
                                 const int32_t* k_h, int32_t k_max, const float* kv_state,
                                 const float* k_state, const double* page_kmean,
                                 const float* g_lin, const float* g_sp, void* o,
                                 int32_t* sel_out, void* stream) {
  hsa_status_t st = check_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state,
                                  k_state, o);
  if (st != HSA_OK) return st;
  if (!page_kmean) return HSA_ERR_INVALID_ARG;
  const size_t need = hsa_forward_noalloc_bytes(cfg, n_q, n_cand, n_cur_pages, k_h, k_max);
  if (need == 0) return HSA_ERR_UNSUPPORTED;
  if (need > (size_t)HSA_NOALLOC_SCRATCH_BYTES) return HSA_ERR_WORKSPACE;
  uint8_t* base = scratch_for_current_device();
  if (!base) return HSA_ERR_DEVICE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = validate_pages(cfg, pool, 0, n_cand + n_cur_pages, s)) != HSA_OK) return st;
  return forward_body(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                      page_kmean, g_lin, g_sp, o, sel_out, base, s);
}

}  // extern "C"

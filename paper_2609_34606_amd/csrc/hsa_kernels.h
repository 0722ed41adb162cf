// Kernel parameter blocks and launch entry points of the HSA library.
// Host-side only; the C ABI (hsa_api.hip) validates arguments, carves the
// workspace and calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/hsa.h"

namespace hsa {

constexpr int HSA_MAX_CHUNKS = HSA_PLAN_MAX_CHUNKS;

// ------------------------------------------------------------ state update
struct StateParams {
  const void* k;            // [num_slots, H, P, d]
  const void* v;            // [num_slots, H, d, P]
  const int32_t* page_table;
  int32_t H, P, num_slots, max_pages;
  int32_t first_page, n_pages;
  int32_t parts;            // parts per page
  int32_t part_len;         // keys per part (multiple of 8)
  int32_t upw;              // units (page x part) per workgroup
  int32_t n_groups;         // workgroups per (b, h)
  float* ws_S;              // [B*H*n_groups, d, d] partial state, [j][i]
  float* ws_z;              // [B*H*n_groups, d]
  double* ws_k;             // [B*H*n_pages*parts, d] partial key sums
};

struct StateReduceParams {
  float* kv_state;          // [B, H, d, d]
  float* k_state;           // [B, H, d]
  double* page_kmean;       // [B, H, max_pages, d]
  const float* ws_S;
  const float* ws_z;
  const double* ws_k;
  int32_t H, P, max_pages, first_page, n_pages, parts, n_groups;
};

hipError_t launch_state_update(int dtype, int d, int B, const StateParams& p,
                               const StateReduceParams& r, hipStream_t s);

// ------------------------------------------------------------ page select
struct QsumParams {
  const void* q;            // [B, n_q, H, d]
  int32_t n_q, HD;          // HD = H * d
  int32_t rows_per_split, n_split;
  double* ws_qs;            // [B, n_split, H*d]
};

struct SelectParams {
  const double* ws_qs;      // [B, n_split, H*d]
  const double* page_kmean; // [B, H, max_pages, d]
  int32_t H, n_q, n_split, max_pages, n_cand, k_max;
  int32_t k_h[HSA_MAX_HEADS];
  int32_t* sel;             // [B, H, k_max]
  double* sel_score;        // nullable
  const int32_t* cand_range;  // [B, 2] candidate pages [lo, hi) of each batch
                              // entry (Stage-1 chunk), nullable: [0, n_cand)
};

// Stage-1 prompt-level retrieval: top-1 chunk by cosine similarity.
struct ChunkSelectParams {
  const float* prompt;      // [B, E]
  const float* chunks;      // [B, M, E]
  const int32_t* chunk_first;  // [B, M + 1] first logical page of each chunk
  int32_t E, M, n_cand;
  int32_t* chunk_out;       // [B] nullable
  double* chunk_score;      // [B] nullable
  int32_t* cand_range;      // [B, 2] pages of the chosen chunk, clamped to [0, n_cand]
};

hipError_t launch_chunk_select(int B, const ChunkSelectParams& p, hipStream_t s);

hipError_t launch_page_select(int dtype, int d, int B, const QsumParams& qp,
                              const SelectParams& sp, hipStream_t s);
// The first stage of launch_page_select alone (fp64 column sums of the query
// rows in splits of qp.rows_per_split).
hipError_t launch_qsum(int dtype, int B, const QsumParams& qp, hipStream_t s);

// ------------------------------------------------------------ block selection
// Key blocks: runs of kBlockHist tokens inside each selected history page and
// of kBlockCur tokens inside each current page (the last block of a page is
// shorter when the block size does not divide P); query blocks: runs of
// kBlockQ queries. Both key block sizes are multiples of the attention
// kernels' 64-key tile, so a block is a whole number of tiles.
constexpr int kBlockQ = 64, kBlockHist = 128, kBlockCur = 64;

struct BlockSelParams {
  const void* k;              // pool keys [num_slots, H, P, d]
  const int32_t* page_table;  // [B, max_pages]
  const int32_t* sel;         // [B, H, k_max] (not read when k_max == 0)
  int32_t H, P, n_q, num_slots, max_pages, k_max, cur_first, n_cur;
  int32_t n_qb;               // query blocks
  int32_t n_qt;               // attention query tiles (two query blocks each)
  int32_t n_blk_max;          // key blocks of the longest list (row length of the buffers below)
  int32_t n_pad;              // n_blk_max rounded up to a power of two, >= 64
  int32_t rpg;                // query blocks per pooled-rows workgroup (1..4)
  int32_t qs_split;           // splits of ws_qs (each kBlockQ / 2 rows)
  double scale;               // pooled-map scale
  double tau_min, tau_max;
  const double* ws_qs;        // [B, qs_split, H*d] query column sums
  double* kbar_t;             // [B, H, d, n_blk_max] block mean keys, d-major
  double* row_c;              // [B, H, n_qb, n_blk_max] cumulative weight, sorted order
  int32_t* row_i;             // [B, H, n_qb, n_blk_max] block id, sorted order
  double* row_g;              // [B, H, n_qb] Gini term of each query block
  int2* blist;                // [B, H, n_qt, blist_cap] tile lists
  int32_t* blist_len;         // [B, H, n_qt]
  int32_t blist_cap;
  // optional outputs (NULL: not written)
  double* gini;               // [B, H]
  double* tau;                // [B, H]
  int32_t* n_kept;            // [B, H, n_qb]
  int32_t* kept;              // [B, H, n_qb, kept_len]
  int32_t kept_len;
  double* pooled;             // [B, H, n_qb, kept_len]
};

// Block means, pooled map, per-row order, Gini terms and cumulative weights,
// then the per-head threshold, the kept prefixes and the tile lists of the
// attention kernel. ws_qs must already hold the query column sums.
hipError_t launch_block_select(int dtype, int d, int B, const BlockSelParams& p, hipStream_t s);
// LDS bytes of one pooled-rows workgroup (at most 64 KB is allowed).
size_t block_rows_lds_bytes(int d, int n_pad, int rpg);

// ------------------------------------------------------------ Linformer compression
struct CompressParams {
  const void* k;              // pool keys [num_slots, H, P, d]
  const void* v;              // pool values [num_slots, H, d, P]
  const int32_t* page_table;  // [B, max_pages]
  const void* e_k;            // [H, R, P]: e_k[h][j][t] = E_K^(h)[t][j]
  const void* e_v;            // [H, R, P]
  void* ck;                   // [num_slots, H, R, d]
  void* cv;                   // [num_slots, H, d, R]
  float* partial;             // [B, H, n_pages, parts, 2, R*d] (parts > 1)
  int32_t H, P, R, D, num_slots, max_pages, first_page, n_pages;
  int32_t parts;              // parts per page
  int32_t part_len;           // tokens per part (multiple of 64)
};

// Compresses logical pages [first_page, first_page + n_pages) of every batch
// entry (bf16: R in {32, 64, 128}; fp32: any R).
hipError_t launch_compress(int dtype, int B, const CompressParams& p, hipStream_t s);

// ------------------------------------------------------------ page append
struct PageWriteParams {
  void* k;                    // pool keys [num_slots, H, P, d]
  void* v;                    // pool values [num_slots, H, d, P]
  const int32_t* page_table;  // [B, max_pages]
  const void* k_src;          // [B, n_pages * P, H, d] token-major
  const void* v_src;          // [B, n_pages * P, H, d]
  const int32_t* src_of;      // [P] stored position -> raster token, NULL: identity
  int32_t H, P, num_slots, max_pages, first_page, n_pages;
};

hipError_t launch_page_write(int dtype, int d, int B, const PageWriteParams& p, hipStream_t s);

// Cube order of a page of T x H x W tokens (see hsa_cube_order in hsa.h):
// src_of[n] = raster index of the token stored at position n. Returns the
// number of positions covered by whole cubes.
int cube_order(int T, int H, int W, int ct, int ch, int cw, int32_t* src_of);

// ------------------------------------------------------------ attention
enum AttnMode : int32_t {
  ATTN_FINAL = 0,   // fused linear branch + gated merge, write o (dtype)
  ATTN_SPARSE = 1,  // write o_sp (fp32) and lse
};

// Work schedule of the bf16 attention kernels, chosen by plan_attention.
struct AttnSchedule {
  // Attention items of one batch entry are numbered head by head in head_order, each head
  // contributing n_split[h] * nqt items (split-major, query tile fastest).
  int32_t nqt;                           // query tiles of 32 * waves queries
  int32_t waves;                         // waves per workgroup (4 or 8)
  int32_t nq32;                          // 32-query wave slots per (head, split): nqt * waves
  int32_t n_items;                       // attention items per batch entry
  int32_t n_order;                       // heads listed in head_order
  int16_t head_order[HSA_MAX_HEADS];
  int32_t item_off[HSA_MAX_HEADS + 1];   // first item of head_order[i]
  int16_t n_split[HSA_MAX_HEADS];        // splits of head h (by head index)
  int16_t list_len[HSA_MAX_HEADS];       // pages the splits of head h cover (<= HSA_MAX_LIST)
  int16_t part_base[HSA_MAX_HEADS];      // first partial slot of head h (n_split > 1)
  int32_t n_part;                        // partial slots per batch entry
  // Items are cut into chunks of consecutive items of one (head, split);
  // XCD x runs chunks [xcd_chunk[x], xcd_chunk[x+1]) in that order.
  int32_t n_chunks;
  int32_t chunk_start[HSA_MAX_CHUNKS];
  int32_t chunk_len[HSA_MAX_CHUNKS];
  int32_t xcd_chunk[9];
  int32_t xcd_items;                     // most items on one XCD
  // heads with n_split > 1 (their query tiles merge the splits at the end)
  int32_t n_chead;
  // Stream-K schedule of the page walk (8 waves): items (one 256-query tile
  // of one head) are numbered b, h, query tile; each has max(1, list_len[h])
  // x tiles-per-page 64-key tiles, head h's first one at sk_head_off[h]
  // within a batch entry (sk_head_off[H]: tiles per entry). The launch's
  // tiles are cut into sk_g ranges, one per workgroup: ranges [0, sk_rm) of
  // sk_q + 1 tiles, then ranges of sk_q. sk_whole = 1: range i is item i
  // whole instead (sk_g = items; sk_q, sk_rm unused).
  int32_t sk_g, sk_q, sk_rm, sk_whole;
  int32_t sk_head_off[HSA_MAX_HEADS + 1];
};

struct AttnParams {
  const void* q;            // [B, n_q, H, d]
  const void* k;            // pool keys
  const void* v;            // pool values (d-major pages)
  const int32_t* page_table;
  const int32_t* sel;       // [B, H, k_max]
  int32_t H, P, n_q, num_slots, max_pages, k_max;
  int32_t cur_first, n_cur;
  float sm_scale;           // softmax scale
  float scale_log2;         // sm_scale * log2(e)
  int32_t mode;
  // final mode
  const float* kv_state;    // [B, H, d, d]
  const float* k_state;     // [B, H, d]
  const float* g_lin;       // [B, n_q, H] nullable, [B, n_q, H, d] with gate_elem
  const float* g_sp;
  int gate_elem;            // gates per (query, head, dim) instead of per (query, head)
  void* o;                  // [B, n_q, H, d] dtype
  const float* o_lin;       // [B, n_q, H, d] fp32 linear-branch output of another
                            // launch; NULL: the kernelised branch from the state
  // sparse mode
  float* o_sp;              // [B, n_q, H, d]
  float* lse;               // [B, H, n_q] nullable
  float* part_o;                         // [B, n_part, nq32, d/32 x 16 registers, 64 lanes]
  float* part_lse;                       // [B, n_part, nq32, 64 lanes]
  int32_t* attn_ctr;                     // [B, H, nqt] arrivals of the splits of each query
                                         // tile (zeroed by the launch)
  // block-sparse mode (blist != NULL): each (b, h, query tile) walks its own
  // list of 64-key tiles, entry {slot * H + h, (tile index << 2) | mask}; mask
  // bit w covers query block 2 * qtile + w (waves 2w, 2w + 1)
  const int2* blist;                     // [B, H, nqt, blist_cap]
  const int32_t* blist_len;              // [B, H, nqt]
  int32_t blist_cap;
  AttnSchedule sc;                       // work schedule of the bf16 kernels
};
// Kernels take AttnParams by value; the kernel-argument segment holds 4 KB.
static_assert(sizeof(AttnParams) <= 3584, "AttnParams must leave room in the 4 KB argument segment");
static_assert(HSA_MAX_LIST <= 32767 && 4 * HSA_MAX_HEADS <= 32767, "per-head schedule fields are int16");

// Work schedule of a bf16 attention launch over B batch entries, H heads of
// head dim d, n_q queries, page size P and list_len[h] pages per head, with
// at most max_part partial slots per batch entry. waves = 8: the page walk's
// stream-K ranges (256-query workgroups, one per CU; split = false keeps
// every item in one range). waves = 4: the tile-list walk (128 queries, two
// workgroups per CU): the split of each head's list and the item order,
// split = false keeping every head whole. Fills p.sc and returns true; false
// if no schedule fits (p.sc is then not written). The last few schedules are
// cached (thread-safe), so a call with the inputs of a recent one costs a
// table lookup.
bool plan_attention(AttnParams& p, int B, int H, int d, int n_q, int P, const int* list_len,
                    int max_part, bool split, int waves);
// Workspace of split key lists for n_part partial slots (any workgroup
// width): partial outputs, then partial LSEs, then the arrival counters.
size_t attention_partial_bytes(int B, int H, int d, int n_q, int n_part);
size_t attention_partial_o_bytes(int B, int d, int n_q, int n_part);
size_t attention_partial_lse_bytes(int B, int n_q, int n_part);

hipError_t launch_attention(int dtype, int d, int B, const AttnParams& p,
                            hipStream_t s);

}  // namespace hsa

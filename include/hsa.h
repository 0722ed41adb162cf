/*
 * hsa.h -- C ABI of the Hybrid Sparse Attention (HSA) forward pass for
 * AMD Instinct MI355X (gfx950).
 *
 * Method: WorldAttention (arxiv 2609.34606). HSA runs two branches over a
 * paged KV cache and merges them per head:
 *   - a linear global branch over the whole history, kept here as a running
 *     kernelised state (feature map elu(x)+1);
 *   - a page selector: each head scores every history page by the scaled dot
 *     product of the chunk's mean query and the page's mean key and keeps its
 *     top-k_h pages (Sec. 3.2, "Stage 2: page-level retrieval");
 *   - exact softmax attention over the selected pages plus the current
 *     chunk's own pages (Sec. 3.3 "Sparse branch"; App. A.1 eq. attention);
 *   - a sigmoid-gated sum of the two branches (Sec. 3.3 "Gated fusion").
 *
 * Conventions shared by every call
 * --------------------------------
 * Pointers named "device" point to GPU memory the caller allocated; the
 * library never allocates, frees or retains them. "host" pointers are read
 * during the call only. Every call is asynchronous on `stream` (a hipStream_t
 * passed as void*; NULL is the null stream) and makes no host synchronisation,
 * except that with environment variable HSA_CHECK=1 the page table is copied
 * back and validated first (synchronising the stream).
 *
 * Errors: calls return an hsa_status_t. Arguments are validated on the host
 * before any launch; on an error nothing is launched and no output is
 * written. Kernels clamp physical slots into [0, num_slots) so that a corrupt
 * page table cannot fault the GPU (results are then meaningless; HSA_CHECK=1
 * reports HSA_ERR_OUT_OF_RANGE instead). A launch failure is HSA_ERR_DEVICE.
 *
 * Shapes: B batch, H heads (1..64), d head dim (64 or 128), P page size
 * (a multiple of 8, >= 8), n_q queries in the chunk. Element type of q, k, v
 * and o is cfg->dtype (bf16 or fp32); statistics are fp32/fp64 as stated.
 *
 * Layouts (row-major, innermost last):
 *   q, o         [B, n_q, H, d]
 *   pool.k       [num_slots, H, P, d]   key pages
 *   pool.v       [num_slots, H, d, P]   value pages, stored d-major
 *   page_table   [B, max_pages] int32   logical page -> physical slot;
 *                logical pages are in age order (0 = oldest)
 *   kv_state     [B, H, d, d] fp32      kv_state[b][h][j][i] = sum_t phi(k_t)[i] v_t[j]
 *   k_state      [B, H, d] fp32         k_state[b][h][i]     = sum_t phi(k_t)[i]
 *   page_kmean   [B, H, max_pages, d] fp64  mean key of each page
 *   g_lin, g_sp  [B, n_q, H] fp32       gate logits (nullable: logit 0), or
 *                [B, n_q, H, d] fp32    with cfg->gate_dims == d (element-wise)
 *   sel          [B, H, k_max] int32    selected logical pages, -1 padded
 */
#ifndef HSA_H_
#define HSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HSA_MAX_HEADS 64
#define HSA_MAX_LIST 1024 /* k_max + n_cur_pages per head */
#define HSA_MAX_CAND 8192 /* history pages a selection can score */
#define HSA_MAX_BLOCKS 4096 /* key blocks of one head's list (adaptive calls) */

/* Block geometry of the head-adaptive sparse branch (Sec. 3.3, granularity
 * of the sparse branch): history pages are cut into blocks of
 * HSA_BLOCK_HIST tokens, the current chunk's pages into blocks of
 * HSA_BLOCK_CUR tokens, the query chunk into blocks of HSA_BLOCK_Q queries
 * (the last block of a page or of the chunk may be shorter). */
#define HSA_BLOCK_Q 64
#define HSA_BLOCK_HIST 128
#define HSA_BLOCK_CUR 64

typedef enum hsa_status {
  HSA_OK = 0,
  HSA_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, empty key set */
  HSA_ERR_UNSUPPORTED = 2, /* valid but not implemented: d, P, H, sizes  */
  HSA_ERR_OUT_OF_RANGE = 3, /* page outside the pool / page table         */
  HSA_ERR_WORKSPACE = 4,   /* workspace NULL or smaller than required    */
  HSA_ERR_DEVICE = 5,      /* a HIP call failed                          */
  HSA_ERR_IO = 6           /* a file read or write of the host tier failed */
} hsa_status_t;

typedef enum hsa_dtype { HSA_DTYPE_BF16 = 0, HSA_DTYPE_F32 = 1 } hsa_dtype_t;

typedef struct hsa_config {
  int32_t batch;     /* B >= 1 */
  int32_t num_heads; /* H in [1, HSA_MAX_HEADS] */
  int32_t head_dim;  /* d in {64, 128} */
  int32_t page_size; /* P >= 8, P % 8 == 0 */
  int32_t dtype;     /* hsa_dtype_t of q, k, v, o */
  float sm_scale;    /* softmax scale; 0 means 1/sqrt(d) (App. A.1 eq. attention) */
  int32_t gate_dims; /* gate logits per element of a head's output row: 0 or 1 means
                        one logit per (query, head) broadcast over d; head_dim means
                        one per (query, head, dim) (Sec. 3.3 "Gated fusion" describes
                        head-level gates applied element-wise); other values are
                        INVALID_ARG */
} hsa_config_t;

typedef struct hsa_kv_pool {
  const void* k;              /* device [num_slots, H, P, d] */
  const void* v;              /* device [num_slots, H, d, P] */
  const int32_t* page_table;  /* device [B, max_pages] */
  int32_t num_slots;
  int32_t max_pages;
} hsa_kv_pool_t;

/* Human-readable name of a status code (static storage). */
const char* hsa_status_string(hsa_status_t status);

/* Device workspace, in bytes, each call needs for the given sizes. The
 * workspace pointer must be 256-byte aligned. Returns 0 on invalid input. */
size_t hsa_state_update_workspace_size(const hsa_config_t* cfg, int32_t n_pages);
size_t hsa_page_select_workspace_size(const hsa_config_t* cfg, int32_t n_q);
size_t hsa_sparse_attn_workspace_size(const hsa_config_t* cfg, int32_t n_q,
                                      int32_t k_max, int32_t n_cur_pages);
size_t hsa_forward_workspace_size(const hsa_config_t* cfg, int32_t n_q,
                                  int32_t k_max, int32_t n_cur_pages);
/* One workspace size for hsa_block_select, hsa_sparse_attn_adaptive and
 * hsa_forward_adaptive. */
size_t hsa_adaptive_workspace_size(const hsa_config_t* cfg, int32_t n_q,
                                   int32_t k_max, int32_t n_cur_pages);

/* Work schedule of the bf16 attention launch (host-only inspection: it
 * launches nothing and needs no device). For per-head list lengths
 * list_len[h] (selected pages + current pages, host array of H entries, each
 * in [1, HSA_MAX_LIST]) and n_q queries it runs the planner that
 * hsa_forward (adaptive = 0) or the tile-list walk of the adaptive calls
 * (adaptive = 1) use, for cfg->batch batch entries. Page walk: writes the
 * work items of one batch entry (256-query tiles x heads), the workgroups
 * of the launch (each walks one of that many equal ranges of the launch's
 * 64-key tiles, at most HSA_PLAN_MAX_CHUNKS; launches of at least
 * 4 x HSA_PLAN_MAX_CHUNKS items, and launches of at most HSA_PLAN_MAX_CHUNKS
 * items whose longest item exceeds a range by at most four tiles, take one
 * workgroup per whole item) and the most pieces the ranges cut an item
 * into. Tile-list walk: the work items (128-query tile x key
 * split), the chunks of the launch's schedule table (at most
 * HSA_PLAN_MAX_CHUNKS) and the largest key split of a head. Each output
 * pointer is nullable. Errors: INVALID_ARG, UNSUPPORTED (no schedule fits;
 * the attention calls then return the same). */
#define HSA_PLAN_MAX_CHUNKS 256
hsa_status_t hsa_attention_plan(const hsa_config_t* cfg, int32_t n_q, const int32_t* list_len,
                                int32_t adaptive, int32_t* n_items, int32_t* n_chunks,
                                int32_t* max_split);

/* Key blocks of a list of n_hist_pages history pages and n_cur_pages current
 * pages: n_hist_pages * ceil(P / HSA_BLOCK_HIST) + n_cur_pages * ceil(P /
 * HSA_BLOCK_CUR). With n_hist_pages = k_max it is the row length of the
 * per-block outputs of hsa_block_select. Returns -1 on invalid input. */
int32_t hsa_block_count(const hsa_config_t* cfg, int32_t n_hist_pages, int32_t n_cur_pages);

/*
 * hsa_state_update -- fold logical pages [first_page, first_page+n_pages) of
 * every batch entry into the linear-branch state and write their page index.
 *
 * Linear state (kernelised running form of the linear branch, Sec. 3.3 with
 * feature map phi = elu + 1): for every key k_t, value v_t of those pages,
 *   kv_state[b][h][j][i] += phi(k_t)[i] * v_t[j],   k_state[b][h][i] += phi(k_t)[i].
 * Page index (Sec. 3.2 Stage 2, "average key" of a page; Sec. 3.2 "L1"
 * holds page indices built from the keys):
 *   page_kmean[b][h][p][:] = (1/P) sum_{t<P} K[slot(p)][h][t][:], in fp64.
 * A cold build is (first_page = 0, n_pages = all pages) on zeroed states; a
 * streaming step folds only the newly written pages. The result does not
 * depend on the launch configuration (fixed-order reductions, no atomics).
 *
 * kv_state, k_state: device fp32, read-modify-write. page_kmean: device fp64,
 * rows outside the range untouched. ws: device workspace of
 * hsa_state_update_workspace_size(cfg, n_pages) bytes. n_pages == 0 is a
 * no-op. Errors: INVALID_ARG (NULL, bad range), OUT_OF_RANGE (range beyond
 * max_pages), UNSUPPORTED (d, P), WORKSPACE.
 */
hsa_status_t hsa_state_update(const hsa_config_t* cfg, const hsa_kv_pool_t* pool,
                              int32_t first_page, int32_t n_pages, float* kv_state,
                              float* k_state, double* page_kmean, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Page append (the page writer of row a1): copies the keys and values of
 * n_pages new pages of every batch entry, token-major as a projection writes
 * them, into their pool slots (logical pages [first_page, first_page +
 * n_pages) through the page table) in the pool's layouts: key pages [P][d],
 * value pages d-major [d][P]. The pool memory (pool->k, pool->v) is written.
 * k_src, v_src: device [B, n_pages * P, H, d] of cfg->dtype, the tokens of
 * each new page in raster order (frame, row, column). src_of: device int32
 * [P] or NULL; stored position i of a page takes token src_of[i] of that
 * page (entries are clamped into [0, P); a permutation is expected), NULL
 * keeps the raster order. With the table of hsa_cube_order, every run of B
 * stored tokens in the whole-cube prefix of a page is one cube, so the key
 * blocks of the head-adaptive calls are cubes. Fold the pages with
 * hsa_state_update afterwards. Errors: INVALID_ARG (NULL, bad range),
 * OUT_OF_RANGE (range beyond max_pages), UNSUPPORTED (d, P).
 */
hsa_status_t hsa_page_write(const hsa_config_t* cfg, const hsa_kv_pool_t* pool, const void* k_src,
                            const void* v_src, int32_t first_page, int32_t n_pages,
                            const int32_t* src_of, void* stream);

/*
 * Cube order of a page of `frames` x `height` x `width` tokens (App. "Block
 * Sparse Attention", the flattening index of (C_t, C_h, C_w) cubes; Sec. 3.3
 * "Inter- and intra-chunk sparse granularity" uses (4, 8, 4) for retrieved
 * history, B = 128, and (4, 4, 4) for the current chunk, B = 64). Host-only.
 * Writes src_of[i] = raster index (t * height + h) * width + w of the token
 * stored at position i, for i < frames * height * width (host int32 array of
 * that length). Cubes that fit whole come first in the paper's order (cube
 * index along t, then h, then w; tokens in (t, h, w) order inside a cube);
 * when the cube does not divide the page (a 480p frame is 30 x 52 tokens:
 * 30 is not a multiple of 8 or 4; a 3-frame chunk is shorter than C_t = 4)
 * the cubes truncated along the far edges follow, in the same order. If the
 * extents are multiples of the cube this is exactly the paper's index.
 * Returns the number of positions covered by whole cubes (a multiple of
 * ct * ch * cw), or -1 on invalid input (non-positive sizes, NULL).
 */
int32_t hsa_cube_order(int32_t frames, int32_t height, int32_t width, int32_t ct, int32_t ch,
                       int32_t cw, int32_t* src_of);

/*
 * hsa_page_select -- Stage-2 page-level retrieval (Sec. 3.2): per batch entry
 * and head h, with qbar the mean of the n_q queries of head h and kbar_p the
 * page's mean key,
 *   alpha_p = qbar . kbar_p / sqrt(d)   for every candidate page p < n_cand,
 * and sel[b][h][0..k_eff) = the k_eff = min(k_h[h], n_cand) candidates in
 * decreasing alpha, equal scores ordered by increasing logical page index;
 * sel[b][h][k_eff..k_max) = -1. All arithmetic is fp64.
 *
 * q: device [B, n_q, H, d] (cfg->dtype). page_kmean: device fp64
 * [B, H, max_pages, d] (rows [0, n_cand) are read). k_h: host int32 [H],
 * each in [0, k_max]. sel: device int32 [B, H, k_max]. sel_score: device fp64
 * [B, H, k_max] or NULL (alpha of each selected page, 0 in padding).
 * n_cand in [0, min(max_pages, HSA_MAX_CAND)]. ws: device workspace of
 * hsa_page_select_workspace_size(cfg, n_q) bytes.
 */
hsa_status_t hsa_page_select(const hsa_config_t* cfg, const void* q, int32_t n_q,
                             const double* page_kmean, int32_t max_pages,
                             int32_t n_cand, const int32_t* k_h, int32_t k_max,
                             int32_t* sel, double* sel_score, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * hsa_sparse_attn -- sparse branch alone (Sec. 3.3; App. A.1 eq. attention
 * with a zero mask on the active keys): per batch entry and head, the active
 * keys are the pages sel[b][h][0..) (up to the first entry outside
 * [0, max_pages)) followed by logical pages [cur_first_page,
 * cur_first_page + n_cur_pages), with all their P tokens (Sec. 3.2 "Active
 * KV construction", here a virtual concatenation through the page table).
 *   o_sp[b][i][h] = sum_j softmax_j(scale * q_i . k_j) v_j   (fp32)
 *   lse[b][h][i]  = log sum_j exp(scale * q_i . k_j)          (nullable)
 * k_h: host int32 [H], upper bounds on the valid entries of each sel row
 * (used for scheduling only; may be NULL meaning k_max). A head whose active
 * set is empty is an error only if n_cur_pages == 0 and k_max == 0
 * (INVALID_ARG); otherwise an empty row of sel with n_cur_pages == 0 yields
 * o_sp = 0 and lse = -inf for that head.
 * ws: hsa_sparse_attn_workspace_size(cfg, n_q, k_max, n_cur_pages) bytes.
 */
hsa_status_t hsa_sparse_attn(const hsa_config_t* cfg, const void* q, int32_t n_q,
                             const hsa_kv_pool_t* pool, const int32_t* sel,
                             int32_t k_max, const int32_t* k_h,
                             int32_t cur_first_page, int32_t n_cur_pages,
                             float* o_sp, float* lse, void* ws, size_t ws_bytes,
                             void* stream);

/*
 * hsa_forward -- the whole HSA forward pass for one chunk:
 *   1. page selection over candidates [0, n_cand) as hsa_page_select;
 *   2. sparse branch over the selected pages plus the current pages
 *      [n_cand, n_cand + n_cur_pages) as hsa_sparse_attn;
 *   3. linear branch from the running state:
 *        O_lin[i] = (sum_a phi(q_i)[a] kv_state[j][a]) / (phi(q_i) . k_state);
 *   4. gated fusion (Sec. 3.3): o = sigmoid(g_lin) O_lin + sigmoid(g_sp) O_sp,
 *      gates broadcast over d (element-wise when cfg->gate_dims == d); a NULL
 *      gate array means logit 0 (weight 1/2).
 * The state and page index must already cover the pages (hsa_state_update
 * over [0, n_cand + n_cur_pages) or its streaming equivalent).
 *
 * o: device [B, n_q, H, d] in cfg->dtype. sel_out: device int32
 * [B, H, k_max] or NULL. k_h: host int32 [H] in [0, k_max]. Errors as
 * above; n_cand + n_cur_pages must be <= max_pages and each head must have at
 * least one active page (n_cur_pages >= 1 or k_h[h] >= 1 with n_cand >= 1).
 * ws: hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages) bytes.
 */
hsa_status_t hsa_forward(const hsa_config_t* cfg, const void* q, int32_t n_q,
                         const hsa_kv_pool_t* pool, int32_t n_cand,
                         int32_t n_cur_pages, const int32_t* k_h, int32_t k_max,
                         const float* kv_state, const float* k_state,
                         const double* page_kmean, const float* g_lin,
                         const float* g_sp, void* o, int32_t* sel_out, void* ws,
                         size_t ws_bytes, void* stream);

/*
 * hsa_forward_selected -- steps 2-4 of hsa_forward for a page selection the
 * caller already holds (for instance from hsa_page_select): the sparse branch
 * over sel[b][h] (entries up to the first one outside [0, max_pages)) plus the
 * current pages [n_cand, n_cand + n_cur_pages), the linear branch and the
 * gated fusion. hsa_forward is hsa_page_select followed by this call.
 * sel: device int32 [B, H, k_max]. k_h: host int32 [H], upper bounds on the
 * valid entries of each row (the work split is planned from them). Other
 * arguments as hsa_forward. ws: hsa_forward_workspace_size(...) bytes.
 */
hsa_status_t hsa_forward_selected(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                  const hsa_kv_pool_t* pool, const int32_t* sel,
                                  int32_t k_max, const int32_t* k_h, int32_t n_cand,
                                  int32_t n_cur_pages, const float* kv_state,
                                  const float* k_state, const float* g_lin, const float* g_sp,
                                  void* o, void* ws, size_t ws_bytes, void* stream);

/*
 * hsa_forward_noalloc -- hsa_forward for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. Same arguments, computation and outputs as hsa_forward,
 * except that there is no ws / ws_bytes: the workspace is a library-owned
 * static device buffer of HSA_NOALLOC_SCRATCH_BYTES bytes. Each GPU the
 * library runs on holds its own copy of that buffer from the first use of
 * the library on it until the process ends. The call allocates nothing and
 * frees nothing (no hipMalloc / hipFree, no allocating library routine).
 *
 * hsa_forward_noalloc_bytes returns the bytes of that buffer a call with
 * these sizes uses (query sums, the selection when sel_out is NULL, and the
 * split partials of the attention schedule it plans), or 0 on invalid input.
 * A call that needs more than HSA_NOALLOC_SCRATCH_BYTES returns
 * HSA_ERR_WORKSPACE without launching (use hsa_forward with a larger
 * workspace then). The buffer keeps the last call's contents; every byte a
 * call reads it first writes in the same call. Calls that overlap on one GPU
 * (on different streams, or from different threads without ordering) share
 * the one buffer and race: serialise them.
 */
#define HSA_NOALLOC_SCRATCH_BYTES (128u << 20)
size_t hsa_forward_noalloc_bytes(const hsa_config_t* cfg, int32_t n_q, int32_t n_cand,
                                 int32_t n_cur_pages, const int32_t* k_h, int32_t k_max);
hsa_status_t hsa_forward_noalloc(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                 const hsa_kv_pool_t* pool, int32_t n_cand, int32_t n_cur_pages,
                                 const int32_t* k_h, int32_t k_max, const float* kv_state,
                                 const float* k_state, const double* page_kmean,
                                 const float* g_lin, const float* g_sp, void* o,
                                 int32_t* sel_out, void* stream);

/*
 * Head-adaptive block-sparse sparse branch (Sec. 3.3 "Sparse branch" and
 * "Head-level sparsity adaptation"; the appendix on the sparse branch defines
 * the pooled map, the coverage rule and the Gini coefficient; Sec. 4.5 fixes
 * (tau_max, tau_min) = (1.00, 0.35)).
 *
 * Per batch entry and head h the active pages are those of hsa_sparse_attn
 * (sel[b][h][0..) up to the first entry outside [0, max_pages), then the
 * current pages), cut into key blocks (HSA_BLOCK_HIST tokens per block in a
 * history page, HSA_BLOCK_CUR in a current page) numbered j = 0..N-1 in list
 * order, block by block inside each page. Query block i holds queries
 * [HSA_BLOCK_Q i, HSA_BLOCK_Q (i+1)) of the chunk. With qbar_i and kbar_j the
 * means of the block's queries and keys and s = sm_scale (0: 1/sqrt(d)):
 *   p_i,j = softmax_j(s * qbar_i . kbar_j)                      (pooled map)
 *   G     = (1/n_qb) sum_i (1/N) sum_m (N - 2m + 1) p_i,(m)      (Gini; p_i,(m)
 *           the m-th largest weight of row i, m = 1..N)
 *   tau   = tau_min + G (tau_max - tau_min)
 * and query block i keeps the shortest prefix of its blocks in the order
 * (weight descending, block id ascending) whose running weight reaches tau
 * (every block if rounding keeps the total below tau, and every block when
 * tau >= 1). All of it is fp64.
 * Query block i then attends exactly to the keys of its kept blocks (App.
 * A.1 eq. attention with a zero mask on them and -inf elsewhere).
 * tau_min, tau_max: 0 <= tau_min <= tau_max <= 1. N must not exceed
 * HSA_MAX_BLOCKS (UNSUPPORTED). Other arguments and errors as hsa_sparse_attn.
 * ws: hsa_adaptive_workspace_size(cfg, n_q, k_max, n_cur_pages) bytes.
 */

/*
 * hsa_block_select -- the block selection alone, for inspection: gini[b][h]
 * = G, tau[b][h] = tau (device fp64 [B, H], nullable), n_kept[b][h][i] the
 * kept count of query block i (device int32 [B, H, n_qb], nullable), kept
 * [b][h][i][0..n_kept) the kept block ids in selection order and -1 after
 * (device int32 [B, H, n_qb, kept_len], nullable), pooled[b][h][i][j] = p_i,j
 * in block order, 0 past N (device fp64 [B, H, n_qb, kept_len], nullable),
 * with n_qb = ceil(n_q / HSA_BLOCK_Q) and kept_len >= hsa_block_count(cfg,
 * k_max, n_cur_pages) when kept or pooled is given.
 */
hsa_status_t hsa_block_select(const hsa_config_t* cfg, const void* q, int32_t n_q,
                              const hsa_kv_pool_t* pool, const int32_t* sel, int32_t k_max,
                              int32_t cur_first_page, int32_t n_cur_pages, double tau_min,
                              double tau_max, double* gini, double* tau, int32_t* n_kept,
                              int32_t* kept, double* pooled, int32_t kept_len, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * hsa_sparse_attn_adaptive -- the block-sparse sparse branch: block selection
 * as above, then for every query i of query block qb
 *   o_sp[b][i][h] = sum_j softmax_j(scale * q_i . k_j) v_j,  lse[b][h][i] = log sum_j exp(...)
 * over the keys j of the blocks qb keeps (fp32 outputs, lse nullable). k_h:
 * host int32 [H] upper bounds on the valid entries of each sel row (the work
 * split is planned from them), or NULL meaning k_max.
 */
hsa_status_t hsa_sparse_attn_adaptive(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                      const hsa_kv_pool_t* pool, const int32_t* sel,
                                      int32_t k_max, const int32_t* k_h, int32_t cur_first_page,
                                      int32_t n_cur_pages, double tau_min, double tau_max,
                                      float* o_sp, float* lse, void* ws, size_t ws_bytes,
                                      void* stream);

/*
 * hsa_forward_adaptive -- hsa_forward with the block-sparse sparse branch:
 * page selection over candidates [0, n_cand), block selection over the
 * selected pages and the current pages [n_cand, n_cand + n_cur_pages), the
 * block-sparse sparse branch, the linear branch and the gated fusion.
 * Arguments and errors as hsa_forward plus the two thresholds.
 */
hsa_status_t hsa_forward_adaptive(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                  const hsa_kv_pool_t* pool, int32_t n_cand,
                                  int32_t n_cur_pages, const int32_t* k_h, int32_t k_max,
                                  double tau_min, double tau_max, const float* kv_state,
                                  const float* k_state, const double* page_kmean,
                                  const float* g_lin, const float* g_sp, void* o,
                                  int32_t* sel_out, void* ws, size_t ws_bytes, void* stream);

/*
 * Two-stage retrieval of the hierarchical KV cache (Sec. 3.2). The KV bank is
 * a sequence of chunks in generation order, chunk m holding the history pages
 * [chunk_first[b][m], chunk_first[b][m+1]) (chunk_first[b][n_chunks] =
 * n_cand), with one prompt embedding per chunk (the chunk index).
 *
 * hsa_chunk_select -- Stage 1, prompt-level retrieval: per batch entry,
 *   cos_m = (p . c_m) / (|p| |c_m|)  (0 when a norm is 0), fp64,
 * and the top-1 chunk m* by (cos desc, m asc). Writes chunk_out[b] = m*
 * (nullable), chunk_score[b] = cos_m* (nullable, fp64) and cand_range[b] =
 * {chunk_first[b][m*], chunk_first[b][m*+1]} clamped to [0, n_cand] (device
 * int32 [B, 2], the Stage-2 candidates). prompt_emb: device fp32 [B, E];
 * chunk_emb: device fp32 [B, n_chunks, E]; chunk_first: device int32
 * [B, n_chunks + 1].
 */
hsa_status_t hsa_chunk_select(const hsa_config_t* cfg, const float* prompt_emb,
                              const float* chunk_emb, int32_t emb_dim, int32_t n_chunks,
                              const int32_t* chunk_first, int32_t n_cand, int32_t* chunk_out,
                              double* chunk_score, int32_t* cand_range, void* stream);

/* Workspace of hsa_forward_retrieval. */
size_t hsa_retrieval_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                    int32_t n_cur_pages);

/*
 * hsa_forward_retrieval -- hsa_forward with Stage 1 in front: the chunk of
 * hsa_chunk_select, then Stage-2 page selection among that chunk's pages only
 * (sel holds logical page indices; a head keeps min(k_h[h], pages of the
 * chunk) pages), the sparse branch over them plus the current pages
 * [n_cand, n_cand + n_cur_pages), the linear branch over the state and the
 * gated fusion. chunk_out: device int32 [B] or NULL. Other arguments and
 * errors as hsa_forward. ws: hsa_retrieval_workspace_size(...) bytes.
 */
hsa_status_t hsa_forward_retrieval(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                   const hsa_kv_pool_t* pool, const float* prompt_emb,
                                   const float* chunk_emb, int32_t emb_dim, int32_t n_chunks,
                                   const int32_t* chunk_first, int32_t n_cand,
                                   int32_t n_cur_pages, const int32_t* k_h, int32_t k_max,
                                   const float* kv_state, const float* k_state,
                                   const double* page_kmean, const float* g_lin,
                                   const float* g_sp, void* o, int32_t* chunk_out,
                                   int32_t* sel_out, void* ws, size_t ws_bytes, void* stream);

/*
 * Host-managed tiers of the KV cache (Sec. 3.2 "Cache hierarchy and
 * dataflow"): L1 = the device pool, L2 = pinned host memory, L3 = a file on
 * a local drive. A tier owns the placement of logical pages: each page
 * (b, p) lives in one of the pool's num_slots slots, one of l2_slots host
 * slots or one of l3_slots file slots, and the tier keeps the device page
 * table's entries of pages in the pool up to date. A slot holds every head
 * of a page. Pages leave the pool least recently used first, only when a slot
 * is needed, and L2 spills to L3 the same way; the pages a fetch lists are in
 * the pool before anything that follows on the same stream. Kernels only
 * touch pages in the pool, so a forward pass over fetched pages gives the
 * same result as one with every page resident. The page index and the linear
 * state cover a page from the moment it is folded (hsa_state_update right
 * after writing it), whatever its tier later.
 *
 * Streams: place, fetch and the kernels that read the pool go on one
 * "compute" stream; a prefetch may go on another stream and then overlaps
 * them. A fetch moves each page with one swap kernel on the calling stream:
 * the page it brings in from pinned host memory and the page it displaces,
 * which goes to the host slot the first one leaves, cross the link in both
 * directions at once, in place. A prefetch (which overlaps compute, so
 * takes no compute units) and place use DMA copies: host-to-device on the
 * calling stream, device-to-host on a stream of the tier's own, the page
 * going out taking the free host slot freed first. The tier orders all of
 * them with events and makes the calling stream wait for its own copies
 * before returning. A move from L2 to L3 or from L3 waits on the host for
 * the copies it depends on (so that call blocks). A tier is not
 * thread-safe.
 *
 * Backup mode (l3_backup != 0): the file holds a copy of every page. Each
 * page owns file slot i from its placement on (i-th page placed), written by
 * the first hsa_tier_commit after the caller has written the page, or when
 * the page leaves L1 and L2 before that; the copy stays. Pages leaving L2
 * then cost no file write, a read from L3 keeps the file copy, and
 * hsa_tier_drop can release every L1 and L2 copy, each page staying
 * restorable from the file.
 */
typedef struct hsa_tier hsa_tier_t;

typedef struct hsa_tier_stats {
  int64_t evictions;  /* pages moved out of L1 (to L2, or to L3 when no L2 slot can take them) */
  int64_t fetches;    /* pages moved into L1 from L2 or L3 (prefetched ones included) */
  int64_t spills;     /* pages moved to L3 from L2 (or from L1 directly) */
  int64_t reloads;    /* pages moved L3 -> L1 */
  int64_t prefetched; /* pages moved into L1 by hsa_tier_prefetch */
  int64_t backups;    /* backup mode: pages written to their own file slot */
} hsa_tier_stats_t;

/* Creates a tier for pool (device k, v, page_table; num_slots L1 slots,
 * max_pages logical pages per batch entry) on the current device.
 * host_k, host_v: pinned host memory (hipHostMalloc; the swap kernel reads
 * and writes it) of l2_slots slots in the pool layout ([l2_slots, H, P, d]
 * and [l2_slots, H, d, P], cfg->dtype), owned by the caller; INVALID_ARG if
 * the device cannot address it. pool->k, pool->v, host_k and host_v 16-byte
 * aligned, else UNSUPPORTED. l3_dir: a directory on the drive where the tier keeps an unnamed
 * file of l3_slots slots (gone when the tier is destroyed); without backup
 * mode l3_slots > 0 needs l2_slots >= 1, with it l3_slots >= 1 (l2_slots may
 * be 0). The tier allocates two pinned staging pages for file reads and
 * writes, an internal stream and its events. pool->k == NULL makes a
 * plan-only tier that issues no copy and touches no file (policy
 * inspection). HSA_ERR_IO if the file cannot be created. */
hsa_status_t hsa_tier_create(const hsa_config_t* cfg, const hsa_kv_pool_t* pool, void* host_k,
                             void* host_v, int32_t l2_slots, const char* l3_dir,
                             int32_t l3_slots, int32_t l3_backup, hsa_tier_t** tier);

/* Waits for the tier's own copies, then frees it. Call it once the kernels
 * that read its pages have finished. */
void hsa_tier_destroy(hsa_tier_t* tier);

/* A pool slot for new logical page `page` of batch entry b (written next by
 * the caller on the same stream); if none is free, the least recently used
 * page moves down a tier. A tier holds at most
 * num_slots + l2_slots + l3_slots - 1 pages (num_slots without lower tiers):
 * one lower-tier slot stays free so that a fetch can always swap; in backup
 * mode at most l3_slots pages. UNSUPPORTED beyond that. Sets the page-table
 * entry. */
hsa_status_t hsa_tier_place(hsa_tier_t* tier, int32_t b, int32_t page, int32_t* slot,
                            void* stream);

/* Brings every listed page into the pool: pages host int32 [B, n_per_batch]
 * logical pages (entries < 0 ignored, e.g. a copy of sel plus the current
 * pages); they become the most recently used and are the pages a later
 * prefetch leaves in place. Waits for the last prefetch first.
 * UNSUPPORTED if they do not fit in the pool at once. */
hsa_status_t hsa_tier_fetch(hsa_tier_t* tier, const int32_t* pages, int32_t n_per_batch,
                            void* stream);

/* As hsa_tier_fetch, on a side stream, for pages a later fetch is expected
 * to list (e.g. the chunk Stage 1 will choose): the copies start once the
 * compute stream has passed the last fetch and overlap the kernels that
 * follow it there; no page the last fetch listed or placed since then
 * moves. The next fetch waits for the prefetch. UNSUPPORTED if those pages
 * and the listed ones do not fit in the pool together. */
hsa_status_t hsa_tier_prefetch(hsa_tier_t* tier, const int32_t* pages, int32_t n_per_batch,
                               void* stream);

/* Backup mode: writes every placed page whose file copy is not written yet
 * to its file slot, after the work already on `stream` (the caller's writes
 * of the pages placed since the last commit). The device-to-host copy of one
 * page overlaps the file write of the one before; the call blocks until the
 * writes are done. INVALID_ARG for a tier without backup mode, IO if a
 * write fails. */
hsa_status_t hsa_tier_commit(hsa_tier_t* tier, void* stream);

/* Backup mode: commits, then releases every L1 and L2 copy once the work
 * already on `stream` is done: each page then lives in its file slot only
 * (hsa_tier_locate gives its L3 code), its page-table entry becomes -1, and
 * the next fetch restores it from the file. For a sequence that is paused
 * (its pool and host slots are free for others) and resumed later.
 * INVALID_ARG for a tier without backup mode. */
hsa_status_t hsa_tier_drop(hsa_tier_t* tier, void* stream);

/* Where a page lives: its pool slot (>= 0), -(i + 2) in L2 slot i,
 * -(l2_slots + i + 2) in L3 slot i, -1 never placed. */
int32_t hsa_tier_locate(const hsa_tier_t* tier, int32_t b, int32_t page);

/* Pages moved between tiers so far. */
void hsa_tier_stats(const hsa_tier_t* tier, hsa_tier_stats_t* stats);

/*
 * Linformer linear branch (Sec. 3.3 "Linear branch"; App. "Linear Branch"):
 * per head h, projections E_K^(h), E_V^(h) in R^{L x r} compress keys and
 * values along the sequence. The sequence is cut into segments of length L
 * that are projected independently and concatenated; here a segment is one
 * page (L = P), so each page is compressed once, when it is written.
 */

/* Workspace of hsa_linformer_compress (0 when none is needed). */
size_t hsa_linformer_compress_workspace_size(const hsa_config_t* cfg, int32_t rank,
                                             int32_t n_pages);

/*
 * hsa_linformer_compress -- for logical pages p in [first_page, first_page +
 * n_pages) of every batch entry and every head h, with slot = page_table[b][p]:
 *   ck[slot][h] = E_K^(h)T K[slot][h]              (rank x d)
 *   cv[slot][h] = (E_V^(h)T V[slot][h])^T           (d x rank, d-major like pool.v)
 * e_k, e_v: device [H, rank, P] in cfg->dtype, e_k[h][j][t] = E_K^(h)[t][j].
 * ck: device [num_slots, H, rank, d], cv: device [num_slots, H, d, rank], in
 * cfg->dtype (bf16: fp32 accumulation, rounded once). rank in {32, 64, 128}
 * (UNSUPPORTED otherwise). The compressed pages are themselves a KV pool of
 * page size rank over the same page table: hsa_sparse_attn on it (cfg with
 * page_size = rank, pool {ck, cv, page_table}) is the Linformer branch over
 * the listed pages. Errors as hsa_state_update. ws:
 * hsa_linformer_compress_workspace_size(cfg, rank, n_pages) bytes.
 */
hsa_status_t hsa_linformer_compress(const hsa_config_t* cfg, const hsa_kv_pool_t* pool,
                                    const void* e_k, const void* e_v, int32_t rank,
                                    int32_t first_page, int32_t n_pages, void* ck, void* cv,
                                    void* ws, size_t ws_bytes, void* stream);

/* Workspace of hsa_forward_linformer. */
size_t hsa_linformer_workspace_size(const hsa_config_t* cfg, int32_t n_q, int32_t k_max,
                                    int32_t n_cur_pages);

/*
 * hsa_forward_linformer -- the HSA forward pass with the paper's two
 * branches: page selection as hsa_forward, the head-adaptive block-sparse
 * sparse branch as hsa_forward_adaptive, and the Linformer linear branch over
 * the compressed versions of the same pages (selected, then current):
 *   O_lin = softmax(scale * Q [ck_p1; ck_p2; ...]^T) [cv_p1^T; cv_p2^T; ...],
 *   o = sigmoid(g_lin) O_lin + sigmoid(g_sp) O_sp   (Sec. 3.3 "Gated fusion").
 * ck, cv: the compressed pool of hsa_linformer_compress, which must cover
 * pages [0, n_cand + n_cur_pages); rank as there. Other arguments and errors
 * as hsa_forward_adaptive (no linear state is read). ws:
 * hsa_linformer_workspace_size(cfg, n_q, k_max, n_cur_pages) bytes.
 */
hsa_status_t hsa_forward_linformer(const hsa_config_t* cfg, const void* q, int32_t n_q,
                                   const hsa_kv_pool_t* pool, const void* ck, const void* cv,
                                   int32_t rank, int32_t n_cand, int32_t n_cur_pages,
                                   const int32_t* k_h, int32_t k_max, double tau_min,
                                   double tau_max, const double* page_kmean, const float* g_lin,
                                   const float* g_sp, void* o, int32_t* sel_out, void* ws,
                                   size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HSA_H_ */

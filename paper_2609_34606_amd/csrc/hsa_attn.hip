// Sparse branch (exact softmax attention over the selected pages plus the
// current chunk) with the linear branch and the gated fusion in the epilogue.
//
// Sec. 3.3 "Sparse branch" with App. A.1 eq. attention (zero mask on the
// active keys); the active keys are the selected pages followed by the
// current pages (Sec. 3.2 "Active KV construction"). The paper materialises
// the active KV with a contiguous copy; here every key row and value group is
// fetched straight from its page through the page table into LDS, so the
// concatenation costs no extra HBM pass.
//
// Two bf16 walks share the tile layout and the epilogue. Both compute the
// transposed score tile S^T = K Q^T with 32x32x16 bf16 MFMAs, so that a lane
// holds 32 scores of a single query (the running max needs one cross-lane
// exchange per tile, the accumulator rescale one multiply per register), and
// the value product O^T += V^T P^T straight from the d-major value pages. Key
// rows are fed to the score MFMA in a permuted order so that the score
// registers of a lane already form the bf16 operand of the value MFMA.
//  * attn_pp_kernel, the page walk: 256 queries of one head per workgroup
//    (8 waves, one workgroup per CU), 64-key tiles in 4 + 4 LDS rings, the
//    score and value halves of the two waves of each SIMD in alternation.
//  * attn_bf16_kernel, the tile-list walk of the block-sparse mode: 128
//    queries (4 waves, two workgroups per CU), a 3-slot key and a 2-slot
//    value ring, all waves in step.
#include <float.h>

#include <algorithm>
#include <mutex>
#include <queue>
#include <utility>
#include <vector>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

constexpr int kWaveQ = 32;    // queries per wave
constexpr int kMaxWaves = 8;  // waves of the widest workgroup
constexpr int kBN = 64;    // keys per tile

template <int D, int kW = 4>
struct AttnLayout {
  static constexpr int kRowK = 2 * D;                  // bytes per key row
  static constexpr int kChunksK = D / 8;               // 16-byte chunks per key row
  static constexpr int kKTile = kBN * kRowK;           // key tile bytes
  static constexpr int kRowV = kBN * 2;                // bytes per value row (64 keys)
  static constexpr int kVTile = D * kRowV;             // value tile bytes
  // key and value tiles in the rings: 3 + 2 (80 KB at d = 128, keys one
  // tile further ahead) for the 4-wave tile-list walk, two workgroups per
  // CU; 4 + 4 (128 KB) for the 8-wave page walk, one per CU
  static constexpr int kKStages = kW == 8 ? 4 : 3;
  static constexpr int kVStages = kW == 8 ? 4 : 2;
  static constexpr int kVBase = kKStages * kKTile;
  static constexpr int kKV = kVBase + kVStages * kVTile;
  static constexpr int kLinHalf = (D / 2) * D * 2 * 2; // half the state rows, hi + lo
  static constexpr int kLin = kLinHalf + D * 4;        // + normaliser
  static constexpr int kBytes = kKV > kLin ? kKV : kLin;
  static constexpr int kRowsPerInstK = 1024 / kRowK;   // key rows per 1-KB load
  static constexpr int kRowsPerInstV = 1024 / kRowV;   // value rows per 1-KB load
  static constexpr int kInstK = kKTile / 1024 / kW;    // key loads per wave
  static constexpr int kInstV = kVTile / 1024 / kW;    // value loads per wave
};

// Swizzles of 16-byte chunks within LDS rows: 16 consecutive rows read at one
// logical chunk land on distinct bank groups.
template <int D>
__device__ __forceinline__ int swz_k(int row) {
  if constexpr (D == 128) return row & 15;
  else return (row >> 1) & 7;
}
__device__ __forceinline__ int swz_v(int row) { return (row >> 1) & 7; }  // 128-byte rows

// Schedule of a block of N (LDS read -> MFMA) pairs: the first kLdsAhead
// reads, then one MFMA and one read alternately, then the last MFMAs. Each
// MFMA's operand is then read kLdsAhead MFMAs before it is needed.
constexpr int kLdsAhead = 4;
template <int N>
__device__ __forceinline__ void pipeline_lds_mfma() {
  __builtin_amdgcn_sched_group_barrier(0x100, kLdsAhead, 0);  // LDS reads
#pragma unroll
  for (int i = 0; i < N - kLdsAhead; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);        // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);        // LDS read
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kLdsAhead, 0);
}

// Score-tile row m holds key perm(m): bits 2 and 3 swapped, so that lane l's
// score registers 0..7 are keys 8*(l/32)+0..7 and 8..15 are 16+8*(l/32)+0..7.
__device__ __forceinline__ int key_perm(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// Gate weight sigmoid(g[i]); a missing gate array means logit 0 (weight 1/2).
__device__ __forceinline__ float gate_w(const float* g, size_t i) {
  return g ? 1.f / (1.f + __expf(-g[i])) : 0.5f;
}

// Output of one (head, 128-query tile) from its normalised sparse-branch
// accumulators (acc * inv_l; lane holds query l%32, dims 32m + 8(r/4) +
// 4(l/32) + r%4) and log-sum-exp. Sparse mode writes O_sp and the LSE;
// final mode adds the linear branch and the gated fusion:
//   O_lin^T = S^T phi(Q)^T / (phi(Q) . z), the state split into bf16 hi + lo
//   parts (~16 bits kept) and staged through LDS in two halves of its rows;
//   o = sigmoid(g_lin) O_lin + sigmoid(g_sp) O_sp, rounded to bf16, with one
//   gate logit per (query, head) or, with gate_elem, per (query, head, dim).
// Every thread of the workgroup must call it (it synchronises); tid is
// threadIdx.x.
template <int D, int NT>
__device__ __forceinline__ void finish(const AttnParams& p, uint8_t* smem, int b, int h, int q_idx,
                                       const u32x4 (&qf)[D / 16], const f32x16 (&acc)[D / 32],
                                       float inv_l, float lse, int tid) {
  using L = AttnLayout<D>;
  constexpr int KK = D / 16, NM = D / 32;
  const int lane = tid & 63, l32 = lane & 31, half = lane >> 5;
  const int H = p.H;
  const bool q_ok = q_idx < p.n_q;
  if (p.mode == ATTN_SPARSE) {
    if (q_ok) {
      float* orow = p.o_sp + (((size_t)b * p.n_q + q_idx) * H + h) * D;
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d0 = 32 * m + 8 * g + 4 * half;
          *reinterpret_cast<f32x4*>(orow + d0) =
              f32x4{acc[m][4 * g] * inv_l, acc[m][4 * g + 1] * inv_l, acc[m][4 * g + 2] * inv_l,
                    acc[m][4 * g + 3] * inv_l};
        }
      if (p.lse && half == 0) p.lse[((size_t)b * H + h) * p.n_q + q_idx] = lse;
    }
    return;
  }
  if (p.o_lin) {
    // linear branch from another launch (Linformer): gated sum only
    if (q_ok) {
      const size_t gi = ((size_t)b * p.n_q + q_idx) * H + h;
      const float wl = p.gate_elem ? 0.f : gate_w(p.g_lin, gi);
      const float wsp = p.gate_elem ? 0.f : gate_w(p.g_sp, gi);
      const float a_sp = wsp * inv_l;
      const float* lrow = p.o_lin + gi * D;
      uint16_t* orow = static_cast<uint16_t*>(p.o) + gi * D;
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d0 = 32 * m + 8 * g + 4 * half;
          const f32x4 l = *reinterpret_cast<const f32x4*>(lrow + d0);
          float v[4];
          if (p.gate_elem) {
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2)
              v[q2] = gate_w(p.g_lin, gi * D + d0 + q2) * l[q2] +
                      gate_w(p.g_sp, gi * D + d0 + q2) * inv_l * acc[m][4 * g + q2];
          } else {
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) v[q2] = wl * l[q2] + a_sp * acc[m][4 * g + q2];
          }
          *reinterpret_cast<u32x2*>(orow + d0) = u32x2{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
        }
    }
    return;
  }
  __syncthreads();  // all waves are done with the shared memory
  constexpr int RH = D / 2;  // state rows per half
  uint8_t* sh = smem;
  uint8_t* sl = smem + RH * D * 2;
  float* zs = reinterpret_cast<float*>(smem + L::kLinHalf);
  if (tid < D) zs[tid] = p.k_state[((size_t)b * H + h) * D + tid];
  const float* st = p.kv_state + ((size_t)b * H + h) * D * D;
  auto stage_state = [&](int hf) {
    for (int e = 4 * tid; e < RH * D; e += 4 * NT) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(st + (size_t)hf * RH * D + e);
      const int j = e / D, i = e % D;
      const int off = j * (2 * D) + (((i >> 3) ^ swz_k<D>(j)) << 4) + (i & 7) * 2;
      const float hx[4] = {x.x, x.y, x.z, x.w};
      uint32_t hw[2], lw[2];
#pragma unroll
      for (int q2 = 0; q2 < 2; ++q2) {
        hw[q2] = pack_bf16(hx[2 * q2], hx[2 * q2 + 1]);
        lw[q2] = pack_bf16(hx[2 * q2] - bf16_lo(hw[q2]), hx[2 * q2 + 1] - bf16_hi(hw[q2]));
      }
      *reinterpret_cast<u32x2*>(sh + off) = u32x2{hw[0], hw[1]};
      *reinterpret_cast<u32x2*>(sl + off) = u32x2{lw[0], lw[1]};
    }
  };
  stage_state(0);
  __syncthreads();
  u32x4 fq[KK];
  float den = 0.f;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const uint32_t w[4] = {qf[kk].x, qf[kk].y, qf[kk].z, qf[kk].w};
    uint32_t o4[4];
#pragma unroll
    for (int q2 = 0; q2 < 4; ++q2) {
      o4[q2] = pack_bf16(phi(bf16_lo(w[q2])), phi(bf16_hi(w[q2])));
      const int d0 = 16 * kk + 8 * half + 2 * q2;
      den = fmaf(bf16_lo(o4[q2]), zs[d0], den);
      den = fmaf(bf16_hi(o4[q2]), zs[d0 + 1], den);
    }
    fq[kk] = u32x4{o4[0], o4[1], o4[2], o4[3]};
  }
  den += __shfl_xor(den, 32);
  const float inv_den = 1.f / den;
  const size_t gi = ((size_t)b * p.n_q + q_idx) * H + h;
  float wl = 0.5f, wsp = 0.5f;
  if (q_ok && !p.gate_elem) {
    wl = gate_w(p.g_lin, gi);
    wsp = gate_w(p.g_sp, gi);
  }
  const float a_lin = wl * inv_den, a_sp = wsp * inv_l;
  uint16_t* orow = q_ok ? static_cast<uint16_t*>(p.o) + (((size_t)b * p.n_q + q_idx) * H + h) * D
                        : nullptr;
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    if (hf == 1) {
      __syncthreads();  // every wave is done with the first half
      stage_state(1);
      __syncthreads();
    }
#pragma unroll
    for (int mm = 0; mm < NM / 2; ++mm) {
      const int m = hf * (NM / 2) + mm;
      f32x16 al = f32x16{0};
      const int row = 32 * mm + l32;  // row within the staged half
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int off = row * (2 * D) + (((2 * kk + half) ^ swz_k<D>(row)) << 4);
        al = mfma32(ld_lds16(sh + off), fq[kk], al);
        al = mfma32(ld_lds16(sl + off), fq[kk], al);
      }
      if (q_ok) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d0 = 32 * m + 8 * g + 4 * half;
          float v[4];
          if (p.gate_elem) {
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2)
              v[q2] = gate_w(p.g_lin, gi * D + d0 + q2) * inv_den * al[4 * g + q2] +
                      gate_w(p.g_sp, gi * D + d0 + q2) * inv_l * acc[m][4 * g + q2];
          } else {
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) v[q2] = a_lin * al[4 * g + q2] + a_sp * acc[m][4 * g + q2];
          }
          *reinterpret_cast<u32x2*>(orow + d0) = u32x2{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
        }
      }
    }
  }
}

// Split-KV merge without a launch of its own. Every split of a (b, h, query
// tile) writes its normalised partial output and log-sum-exp (wave slot
// cell0 + split * nq32), then counts itself in at the tile's counter; the
// workgroup that arrives last reads all splits back and merges them in split
// order, and returns true; the others return false. The merged sums of the
// partials weighted by exp(lse_s - max), the reciprocal of the weight sum
// and the merged LSE replace acc / inv_l / lse, as the epilogue expects. The
// result does not depend on the order of arrival. Every thread of the
// workgroup must call it; tid is threadIdx.x.
// The splits of a tile may run on different XCDs, whose L2 caches are not
// coherent with each other. The partials therefore go through device-scope
// (agent) atomic stores and loads, which write through to and read from the
// device's point of coherence, instead of fences that would write back and
// invalidate a whole L2: each split waits for its stores to complete before
// it counts itself in, and the last one reads them after its count.
template <int D, typename CellOf>
__device__ __forceinline__ bool last_split_merge(const AttnParams& p, CellOf cell_of, int split, int ns,
                                                 size_t ctr, int tid, f32x16 (&acc)[D / 32],
                                                 float& inv_l, float& lse, uint8_t* smem) {
  const int lane = tid & 63;
  constexpr int NM = D / 32;
  // partial layout per wave slot (cell_of(s): the slot of split s):
  // [accumulator register (NM x 16)][lane], so that every 4-byte access
  // instruction covers 256 contiguous bytes
  auto po = [&](int s) { return p.part_o + cell_of(s) * (NM * 16 * 64) + lane; };
  auto pl = [&](int s) { return p.part_lse + cell_of(s) * 64 + lane; };
  {
    float* o = po(split);
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        __hip_atomic_store(o + (m * 16 + r) * 64, acc[m][r] * inv_l, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(pl(split), lse, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  wait_vmcnt<0>();  // this thread's partial has reached the point of coherence
  // the walk's LDS is free once every wave is here: its first word carries
  // the arrival verdict (a separate shared variable would push the 80 KB
  // tile-list kernel past two workgroups per CU)
  __syncthreads();
  int* s_last = reinterpret_cast<int*>(smem);
  if (tid == 0)
    *s_last = __hip_atomic_fetch_add(p.attn_ctr + ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == ns - 1;
  __syncthreads();
  if (!*s_last) return false;
  auto ld = [](const float* q) { return __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); };
  // the largest split LSE, four loads in flight at a time
  float lmax = -INFINITY;
  for (int s0 = 0; s0 < ns; s0 += 4) {
    float l4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) l4[j] = ld(pl(min(s0 + j, ns - 1)));
#pragma unroll
    for (int j = 0; j < 4; ++j) lmax = fmaxf(lmax, l4[j]);
  }
  auto weight = [&](float ls) { return ls == -INFINITY ? 0.f : __expf(ls - lmax); };
  // sum over the splits in split order of weight x partial, each split's
  // partial and LSE loaded in one batch; this split's partial is taken from
  // its registers, rounded as it was stored, so that the sum does not depend
  // on which split arrives last
  float wsum = 0.f;
  f32x16 before[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) before[m] = f32x16{0};
  auto add_split = [&](int s, f32x16 (&into)[NM]) {
    const float ls = ld(pl(s));
    f32x16 o[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[m][r] = ld(po(s) + (m * 16 + r) * 64);
    const float w = weight(ls);
    wsum += w;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) into[m][r] = fmaf(w, o[m][r], into[m][r]);
  };
  for (int s = 0; s < split; ++s) add_split(s, before);
  {
    const float w = weight(lse);
    wsum += w;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][r] = fmaf(w, acc[m][r] * inv_l, before[m][r]);
  }
  for (int s = split + 1; s < ns; ++s) add_split(s, acc);
  inv_l = wsum > 0.f ? 1.f / wsum : 0.f;
  lse = wsum > 0.f ? lmax + __logf(wsum) : -INFINITY;
  return true;
}

// Zeroes the arrival counters of a launch's split tiles.
__global__ __launch_bounds__(256) void zero_counters_kernel(int32_t* ctr, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) ctr[i] = 0;
}

// The tile-list walk (block-sparse mode): each (b, h, 128-query tile) walks
// its own list of 64-key tiles; waves of a 64-query block that does not
// keep a tile skip its MFMAs and softmax.
template <int D, bool kSmallP, int kW>
__global__ __launch_bounds__(64 * kW, 8 / kW) void attn_bf16_kernel(AttnParams p) {
  static_assert(kW == 4, "tile lists mark two 64-query blocks per workgroup");
  using L = AttnLayout<D, kW>;
  // the kernel's only LDS: two workgroups per CU (160 KB) must fit, or the
  // compiler targets one wave per SIMD and spreads into the AGPRs
  static_assert(2 * L::kBytes <= 160 * 1024, "two tile-list workgroups per CU");
  constexpr int kBM = kWaveQ * kW;
  constexpr int KK = D / 16;   // 16-wide d slices
  constexpr int NM = D / 32;   // 32-wide d blocks of the output
  __shared__ __attribute__((aligned(1024))) uint8_t smem[L::kBytes];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int l32 = lane & 31, half = lane >> 5;
  const int H = p.H, P = p.P;
  const int nqt = p.sc.nqt;
  const int b = blockIdx.y;
  int qtile, h, split;
  {
    // Workgroups go to the 8 XCDs round-robin by id (gridDim.x = 8 *
    // xcd_items, so blockIdx.x % 8 is the XCD). Each XCD runs its own list
    // of chunks of consecutive items of one (head, split): query tiles that
    // read the same pages share them through one L2 instead of every XCD
    // fetching every head.
    const int w = blockIdx.x, x = w & 7;
    int k = w >> 3, c = p.sc.xcd_chunk[x];
    const int c_end = p.sc.xcd_chunk[x + 1];
    while (c < c_end && k >= p.sc.chunk_len[c]) {
      k -= p.sc.chunk_len[c];
      ++c;
    }
    if (c >= c_end) return;
    const int item = p.sc.chunk_start[c] + k;
    int oh = 0;
    while (oh + 1 < p.sc.n_order && p.sc.item_off[oh + 1] <= item) ++oh;
    h = p.sc.head_order[oh];
    const int local = item - p.sc.item_off[oh];
    split = local / nqt;
    qtile = local % nqt;
  }
  const int ns = p.sc.n_split[h];

  // ---- key walk: the (b, h, query tile)'s own list of tiles, each with the
  // query blocks that attend to it; this item's share is split `split` of
  // n_split[h] near-equal parts of the list.
  int u0 = 0, u1, ntiles;
  const int2* lst;
  {
    const size_t cell = ((size_t)b * H + h) * nqt + qtile;
    const int len = ld_const(p.blist_len + cell);
    lst = p.blist + cell * p.blist_cap;
    u1 = len;
    if (ns > 1) {
      const int base = len / ns, rem = len % ns;
      u0 = split * base + min(split, rem);
      u1 = u0 + base + (split < rem ? 1 : 0);
    }
    ntiles = u1 - u0;
  }

  // ---- Q fragment: lane holds query (l%32) of this wave, d = 16kk + 8*half + 0..7
  const uint16_t* qb = static_cast<const uint16_t*>(p.q);
  const int q_idx = qtile * kBM + wave * kWaveQ + l32;
  const int q_ld = min(q_idx, p.n_q - 1);
  u32x4 qf[KK];
  {
    const uint16_t* qrow = qb + (((size_t)b * p.n_q + q_ld) * H + h) * D + 8 * half;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = ld_global16(qrow + 16 * kk);
  }

  const uint16_t* kpool = static_cast<const uint16_t*>(p.k);
  const uint16_t* vpool = static_cast<const uint16_t*>(p.v);

  // Per-lane byte offsets of the tile loads, fixed for the whole walk: key
  // rows (16-byte chunk c of row r) and value rows (8 keys at chunk c of
  // d-row r). A partial tile at the end of a page re-reads its last valid
  // row/group instead of reading past the page.
  auto k_row = [&](int n) { return (wave * L::kInstK + n) * L::kRowsPerInstK + lane / L::kChunksK; };
  auto v_row = [&](int n) { return (wave * L::kInstV + n) * L::kRowsPerInstV + (lane >> 3); };
  auto v_col = [&](int n) { return 8 * ((lane & 7) ^ swz_v(v_row(n))); };
  uint32_t k_off[L::kInstK], v_off[L::kInstV];
#pragma unroll
  for (int n = 0; n < L::kInstK; ++n) {
    const int r = k_row(n);
    k_off[n] = (uint32_t)(r * D + 8 * ((lane % L::kChunksK) ^ swz_k<D>(r))) * 2u;
  }
#pragma unroll
  for (int n = 0; n < L::kInstV; ++n) v_off[n] = (uint32_t)(v_row(n) * P + v_col(n)) * 2u;

  // Load cursors: keys run two tiles ahead of the tile being computed
  // (3-slot ring), values one tile ahead (2-slot ring). The last tile of a
  // page (P not a multiple of 64) loads the 64-key window that ends at the
  // page end: every load is then a scalar page base plus the constant
  // per-lane offsets, with no branch, and the window's leading rows (keys
  // of the previous tile) are masked. Pages shorter than a tile (kSmallP)
  // clamp per lane instead. Past the last tile a cursor stays on it: the
  // extra loads re-read it into ring slots nobody reads, so that every tile
  // issues and waits alike; they are drained before the epilogue.
  auto window = [&](int t) { return kSmallP ? t * kBN : min(t * kBN, P - kBN); };
  auto load_k = [&](int buf, const char* src) {
    uint8_t* dst = smem + buf * L::kKTile + wave * L::kInstK * 1024;
#pragma unroll
    for (int n = 0; n < L::kInstK; ++n) {
      uint32_t off = k_off[n];
      if constexpr (kSmallP) off -= (uint32_t)(max(0, k_row(n) - (P - 1)) * D * 2);
      g2lds16_hidden(src + off, dst + n * 1024);
    }
  };
  auto load_v = [&](int buf, const char* src) {
    uint8_t* dst = smem + L::kVBase + buf * L::kVTile + wave * L::kInstV * 1024;
#pragma unroll
    for (int n = 0; n < L::kInstV; ++n) {
      uint32_t off = v_off[n];
      if constexpr (kSmallP) off -= (uint32_t)(max(0, v_col(n) - (P - 8)) * 2);
      g2lds16_hidden(src + off, dst + n * 1024);
    }
  };
  // the tile of entry e; entries past the item's range repeat its last tile
  // (loads into ring slots nobody reads)
  auto entry = [&](int u) { return ld_const(lst + min(u, u1 - 1)); };
  auto issue_k_at = [&](int buf, int2 e) {
    load_k(buf, reinterpret_cast<const char*>(kpool) + ((size_t)e.x * P + window(e.y >> 2)) * D * 2);
  };
  auto issue_v_at = [&](int buf, int2 e) {
    load_v(buf, reinterpret_cast<const char*>(vpool) + (size_t)e.x * D * P * 2 + (size_t)window(e.y >> 2) * 2);
  };

  f32x16 acc[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) acc[m] = f32x16{0};
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = p.scale_log2;
  const int krow = key_perm(l32);

  // prologue: K(0), V(0), K(1). The entries of the tile being computed (ec),
  // of the next value issue (ev) and of the next key issue (ek) sit in
  // scalar registers, read one iteration ahead.
  constexpr int SK = L::kKStages, SV = L::kVStages;
  static_assert(SV == 2, "the tile-list walk keeps three entries");
  int2 ec = make_int2(0, 0), ev = ec, ek = ec;
  if (ntiles > 0) {
    ec = entry(u0);
    ev = entry(u0 + 1);
    issue_k_at(0, ec);
    issue_v_at(0, ec);
    issue_k_at(1, ev);
    ek = entry(u0 + 2);
    // the query fragments have landed once the three tile copies alone may
    // be outstanding
    wait_vmcnt<2 * L::kInstK + L::kInstV>();
  }
  // Pinned here, on every path into the walk, the query fragments count as
  // loaded for the compiler (which does not see the tile copies). Pinned
  // inside the branch above, the path that skips the walk would leave their
  // loads pending at the join, and the compiler would then wait for every
  // outstanding load, the ring's tile copies included, inside each tile's
  // score products.
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) asm volatile("" : "+v"(qf[kk]));
  // ring slots: kbuf / vbuf of the tile being computed, and of the tiles
  // issued in this iteration (tile + SK - 1 and tile + SV - 1)
  int kbuf = 0, vbuf = 0;
  int kbuf_in = SK - 1, vbuf_in = SV - 1;
  for (int tile = 0; tile < ntiles; ++tile) {
    // K(tile) and V(tile) have landed once at most the loads issued after
    // V(tile) are outstanding: K(tile+1), and one V and one K per later
    // iteration
    wait_vmcnt<L::kInstK + (SV - 2) * (L::kInstK + L::kInstV)>();
    lds_barrier();
    issue_v_at(vbuf_in, ev);
    issue_k_at(kbuf_in, ek);
    // waves of a query block that does not keep this tile skip it
    const int tc = ec.y >> 2;
    const bool active = (ec.y >> (wave >> 1)) & 1;
    if (active) {
      // S^T = K Q^T for the two 32-key halves of the tile: the two MFMA chains
      // alternate, and the key fragments are read from LDS kLdsAhead MFMAs
      // before their use (an LDS read takes several MFMA durations).
      f32x16 s[2];
      {
        const uint8_t* kt_l = smem + kbuf * L::kKTile;
        s[0] = f32x16{0};
        s[1] = f32x16{0};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const int row = 32 * h2 + krow;
            const int chunk = 2 * kk + half;
            const u32x4 a = ld_lds16(kt_l + row * L::kRowK + ((chunk ^ swz_k<D>(row)) << 4));
            s[h2] = mfma32(a, qf[kk], s[h2]);
          }
        pipeline_lds_mfma<2 * KK>();
      }
      // The last tile of a page: window rows holding keys outside the tile
      // are masked (leading rows of the page-end window, or rows past the page
      // for pages shorter than a tile). The empty asm keeps this a real branch:
      // the compiler would otherwise apply the selects to every tile.
      const int nv = min(kBN, P - tc * kBN);
      if (nv < kBN) {
        asm volatile("" ::: "memory");
        const int lo = kSmallP ? 0 : kBN - nv, hi = kSmallP ? nv : kBN;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = 32 * h2 + 16 * (r >> 3) + 8 * half + (r & 7);
            if (key < lo || key >= hi) s[h2][r] = -INFINITY;
          }
      }
      // Online softmax against a reference max m_run (raw score units) that
      // only moves when some score exceeds it by more than 8 in exp2 units:
      // exponentials stay <= 256 and the final normalisation by the row sum
      // is exact for any reference. The test uses each lane's own 32 scores;
      // only when it fires are the two lane halves of a query combined.
      float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
      for (int r = 2; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[1][r]);
      if (__any(mx * c2 > m_run * c2 + 8.f)) {
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const bool grow = mx * c2 > m_run * c2 + 8.f;
        const float m_new = grow ? mx : m_run;
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
        l_run *= alpha;
#pragma unroll
        for (int m = 0; m < NM; ++m) acc[m] *= alpha;
        m_run = m_new;
      }
      const float mc = m_run * c2;
      float rs = 0.f;
      u32x4 pb[4];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        float pv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          pv[r] = __builtin_amdgcn_exp2f(fmaf(s[h2][r], c2, -mc));
          rs += pv[r];
        }
#pragma unroll
        for (int g = 0; g < 2; ++g)
          pb[2 * h2 + g] =
              u32x4{pack_bf16(pv[8 * g + 0], pv[8 * g + 1]), pack_bf16(pv[8 * g + 2], pv[8 * g + 3]),
                    pack_bf16(pv[8 * g + 4], pv[8 * g + 5]), pack_bf16(pv[8 * g + 6], pv[8 * g + 7])};
      }
      l_run += rs;
      // O^T += V^T P^T (NM independent chains), value fragments read ahead
      {
        const uint8_t* vt_l = smem + L::kVBase + vbuf * L::kVTile;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int chunk = 2 * ks + half;
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            const int row = 32 * m + l32;
            const u32x4 a = ld_lds16(vt_l + row * L::kRowV + ((chunk ^ swz_v(row)) << 4));
            acc[m] = mfma32(a, pb[ks], acc[m]);
          }
        }
        pipeline_lds_mfma<4 * NM>();
      }
    }
    {
      // the key entry of tile + 3, read after this tile's LDS traffic so that
      // the scalar load never shares the LDS counter with the operand reads
      __builtin_amdgcn_sched_barrier(0);
      const int2 en = entry(u0 + tile + 3);
      ec = ev;
      ev = ek;
      ek = en;
    }
    kbuf = kbuf == SK - 1 ? 0 : kbuf + 1;
    vbuf = vbuf == SV - 1 ? 0 : vbuf + 1;
    kbuf_in = kbuf_in == SK - 1 ? 0 : kbuf_in + 1;
    vbuf_in = vbuf_in == SV - 1 ? 0 : vbuf_in + 1;
  }
  wait_vmcnt<0>();  // the trailing re-reads

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
  float lse = l_tot > 0.f ? m_run * p.sm_scale + __logf(l_tot) : -INFINITY;
  if (ns > 1) {
    const size_t cell0 = ((size_t)b * p.sc.n_part + p.sc.part_base[h]) * p.sc.nq32 + qtile * kW + wave;
    const size_t cstride = (size_t)p.sc.nq32;
    if (!last_split_merge<D>(p, [&](int s) { return cell0 + (size_t)s * cstride; }, split, ns,
                             ((size_t)b * H + h) * nqt + qtile, (int)threadIdx.x, acc, inv_l, lse, smem))
      return;
  }
  finish<D, 64 * kW>(p, smem, b, h, q_idx, qf, acc, inv_l, lse, (int)threadIdx.x);
}

// Page walk of the selected pages plus the current pages: 256 queries of one
// head per workgroup (8 waves of 32 queries; waves w and w + 4 share a SIMD),
// one workgroup per CU. Each 64-key tile t is two phases per wave:
//   X(t): the scores S(t)^T = K(t) Q^T (16 MFMAs at d = 128, key fragments
//         read from LDS eight ahead);
//   Y(t): the softmax of S(t) and the value product O^T += V(t)^T P(t)^T; the
//         four MFMAs of each 16-key group go out as soon as its P fragment is
//         packed and run under the next group's exponentials.
// Waves 0-3 run X in even slots and Y in odd ones, waves 4-7 the other way
// round, with a workgroup barrier between slots. So in every slot each SIMD
// receives the MFMAs of both its waves and the exponentials of one, and all
// eight waves read LDS (a loaded LDS needs many reads in flight: four
// waves alone return a fraction of its bandwidth). Key and value tiles sit in
// 4-slot rings (128 KB at d = 128) filled by global-to-LDS copies that every
// wave issues for its share right after a barrier.
//
// Stream-K schedule: the tiles of all items of the launch (item = one
// (b, h, 256-query tile), ordered b, h, query tile; list pages x tiles per
// page each) are cut into sk_g equal contiguous ranges, one per workgroup,
// consecutive ranges on one XCD. A workgroup walks the item segments of its
// range in order; an item cut by range boundaries is finished by the last of
// its pieces to arrive, which merges the pieces' partials in piece order.
// A workgroup's first and last segments are the only ones that can be
// pieces; their partials go to its two slots (first: 0, last: 1). Launches
// of many items (sk_whole) take one whole item per workgroup instead: the
// hardware dispatcher balances them, and the workgroups that run on an XCD
// at one time hold consecutive items, which share their pages in its L2.
template <int D, bool kSmallP>
__global__ __launch_bounds__(512, 1) void attn_pp_kernel(AttnParams p_arg) {
  using L = AttnLayout<D, 8>;
  constexpr int kBM = 256;
  constexpr int KK = D / 16;   // 16-wide d slices
  constexpr int NM = D / 32;   // 32-wide d blocks of the output
  __shared__ __attribute__((aligned(1024))) uint8_t smem[L::kBytes];
  using ArgParams = const __attribute__((address_space(4))) AttnParams;

  // workgroup blockIdx.x runs on XCD x = blockIdx.x % 8, which holds
  // G / 8 workgroups (one more for x < G % 8); the ranges of an XCD are
  // contiguous
  auto range_id = [](const AttnSchedule& sc) {
    const int G = sc.sk_g, x = (int)(blockIdx.x & 7);
    return x * (G >> 3) + min(x, G & 7) + (int)(blockIdx.x >> 3);
  };
  // ranges [0, sk_rm) hold sk_q + 1 tiles, the others sk_q
  auto range_start = [](const AttnSchedule& sc, int i) { return i * sc.sk_q + min(i, sc.sk_rm); };
  auto range_of = [](const AttnSchedule& sc, int t) {
    const int big = sc.sk_rm * (sc.sk_q + 1);
    return t < big ? t / (sc.sk_q + 1) : sc.sk_rm + (t - big) / sc.sk_q;
  };
  // item i's first tile (whole-item schedule: range i is item i)
  auto item_start = [](const AttnSchedule& sc, int H, int i) {
    const int per_bh = H * sc.nqt, bb = i / per_bh, hh = (i - bb * per_bh) / sc.nqt;
    const int qt = i - bb * per_bh - hh * sc.nqt;
    const int len = (sc.sk_head_off[hh + 1] - sc.sk_head_off[hh]) / sc.nqt;  // tiles per item of hh
    return bb * sc.sk_head_off[H] + sc.sk_head_off[hh] + qt * len;
  };
  int t_seg, t_end;
  if (p_arg.sc.sk_whole) {
    t_seg = item_start(p_arg.sc, p_arg.H, range_id(p_arg.sc));
    t_end = item_start(p_arg.sc, p_arg.H, range_id(p_arg.sc) + 1);
  } else {
    t_seg = range_start(p_arg.sc, range_id(p_arg.sc));
    t_end = range_start(p_arg.sc, range_id(p_arg.sc) + 1);
  }
  for (; t_seg < t_end;) {
  __syncthreads();  // the previous segment is done with the LDS
  // The segment reads the parameters (through the kernel-argument segment)
  // and the lane's index through values the compiler cannot see through:
  // otherwise it hoists out of the loop the loads and offsets that only the
  // epilogue needs and keeps them live across the walk, which has no scalar
  // or vector registers to spare for them.
  ArgParams* pa = (ArgParams*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(pa));
  const AttnParams& p = *(const AttnParams*)pa;
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63, l32 = lane & 31, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool first = wave < 4;  // matrix phase in even slots
  const int H = p.H, P = p.P;
  const int nqt = p.sc.nqt;
  const int tpp = (P + kBN - 1) / kBN;
  const int per_b = p.sc.sk_head_off[H];
  const int b = t_seg / per_b;
  const int tb = t_seg - b * per_b;
  int h = 0;
  while (h + 1 < H && p.sc.sk_head_off[h + 1] <= tb) ++h;
  // (an empty list still takes one tile of the range: its item writes zeros)
  const int n_tiles_item = std::max(1, (int)p.sc.list_len[h]) * tpp;
  const int ih = tb - p.sc.sk_head_off[h];
  const int qtile = ih / n_tiles_item;
  const int a = ih % n_tiles_item;   // this segment: tiles [a, e) of the item
  const int item0 = t_seg - a;
  const int e = std::min(n_tiles_item, t_end - item0);
  t_seg = item0 + e;
  // Tile v of the item is key tile (v + sigma) mod n_tiles_item of its list.
  // sigma puts the item's largest piece in step with its range: there key
  // tile = tiles since the range start (mod the item's tiles), as for every
  // item that a range holds whole. So the workgroups of one head walk about
  // the same key tiles at the same time and find them in the L2 cache, where
  // unrotated pieces would start anywhere in the list.
  int sigma = 0;
  if (!p.sc.sk_whole) {
    const int r0 = range_of(p.sc, item0), s1 = range_start(p.sc, r0 + 1);
    const int n = n_tiles_item;
    int rs = s1;  // the second piece: larger than the first, or a whole range
    if (item0 + n <= s1 || (item0 + n <= range_start(p.sc, r0 + 2) && s1 - item0 >= item0 + n - s1))
      rs = range_start(p.sc, r0);
    sigma = (item0 - rs) % n;
    if (sigma < 0) sigma += n;
  }

  const int32_t* selrow = p.sel + ((size_t)b * H + h) * p.k_max;
  const int32_t* ptrow = p.page_table + (size_t)b * p.max_pages;
  int n_sel = 0;
  while (n_sel < p.k_max && n_sel + p.n_cur < p.sc.list_len[h]) {
    const int e2 = ld_const(selrow + n_sel);
    if (e2 < 0 || e2 >= p.max_pages) break;
    ++n_sel;
  }
  auto head_of = [&](int li) -> size_t {
    const int lp = li < n_sel ? ld_const(selrow + li) : p.cur_first + (li - n_sel);
    return (size_t)clampi(ld_const(ptrow + lp), 0, p.num_slots - 1) * H + h;
  };
  // The segment's key tiles: [S, S + e - a) mod n_tiles_item, less those
  // beyond the real list's n_real tiles (a selection row may hold fewer
  // pages than the bound the ranges were cut from). The walk starts at k0
  // and wraps from the real list's last tile to its first.
  const int n_list = n_sel + p.n_cur;
  int ntiles, k0;
  {
    const int n = n_tiles_item, n_real = n_list * tpp, len = e - a;
    const int S = a + sigma < n ? a + sigma : a + sigma - n;
    const int c1 = std::max(0, std::min(S + len, n_real) - S);
    const int c2 = S + len > n ? std::min(S + len - n, n_real) : 0;
    ntiles = c1 + c2;
    k0 = c1 > 0 ? S : 0;
  }
  const int pg0 = ntiles > 0 ? k0 / tpp : 0;

  const uint16_t* qb = static_cast<const uint16_t*>(p.q);
  const int q_idx = qtile * kBM + wave * kWaveQ + l32;
  const int q_ld = min(q_idx, p.n_q - 1);
  u32x4 qf[KK];
  {
    const uint16_t* qrow = qb + (((size_t)b * p.n_q + q_ld) * H + h) * D + 8 * half;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = ld_global16(qrow + 16 * kk);
  }
  const uint16_t* kpool = static_cast<const uint16_t*>(p.k);
  const uint16_t* vpool = static_cast<const uint16_t*>(p.v);

  auto k_row = [&](int n) { return (wave * L::kInstK + n) * L::kRowsPerInstK + lane / L::kChunksK; };
  auto v_row = [&](int n) { return (wave * L::kInstV + n) * L::kRowsPerInstV + (lane >> 3); };
  auto v_col = [&](int n) { return 8 * ((lane & 7) ^ swz_v(v_row(n))); };
  uint32_t k_off[L::kInstK], v_off[L::kInstV];
#pragma unroll
  for (int n = 0; n < L::kInstK; ++n) {
    const int r = k_row(n);
    k_off[n] = (uint32_t)(r * D + 8 * ((lane % L::kChunksK) ^ swz_k<D>(r))) * 2u;
  }
#pragma unroll
  for (int n = 0; n < L::kInstV; ++n) v_off[n] = (uint32_t)(v_row(n) * P + v_col(n)) * 2u;

  auto window = [&](int t) { return kSmallP ? t * kBN : min(t * kBN, P - kBN); };
  int kli = pg0, kt = ntiles > 0 ? k0 % tpp : 0, vli = pg0, vt = kt;
  const char* kbase =
      reinterpret_cast<const char*>(kpool) + (ntiles > 0 ? head_of(pg0) : 0) * (size_t)P * D * 2;
  const char* vbase =
      reinterpret_cast<const char*>(vpool) + (ntiles > 0 ? head_of(pg0) : 0) * (size_t)D * P * 2;
  auto load_k = [&](int buf, const char* src) {
    uint8_t* dst = smem + buf * L::kKTile + wave * L::kInstK * 1024;
#pragma unroll
    for (int n = 0; n < L::kInstK; ++n) {
      uint32_t off = k_off[n];
      if constexpr (kSmallP) off -= (uint32_t)(max(0, k_row(n) - (P - 1)) * D * 2);
      g2lds16_hidden(src + off, dst + n * 1024);
    }
  };
  auto load_v = [&](int buf, const char* src) {
    uint8_t* dst = smem + L::kVBase + buf * L::kVTile + wave * L::kInstV * 1024;
#pragma unroll
    for (int n = 0; n < L::kInstV; ++n) {
      uint32_t off = v_off[n];
      if constexpr (kSmallP) off -= (uint32_t)(max(0, v_col(n) - (P - 8)) * 2);
      g2lds16_hidden(src + off, dst + n * 1024);
    }
  };
  auto issue_k = [&](int buf) {
    load_k(buf, kbase + (size_t)window(kt) * D * 2);
    if (kt + 1 < tpp) {
      ++kt;
    } else {
      kt = 0;
      kli = kli + 1 < n_list ? kli + 1 : 0;
      kbase = reinterpret_cast<const char*>(kpool) + head_of(kli) * (size_t)P * D * 2;
    }
  };
  auto issue_v = [&](int buf) {
    load_v(buf, vbase + (size_t)window(vt) * 2);
    if (vt + 1 < tpp) {
      ++vt;
    } else {
      vt = 0;
      vli = vli + 1 < n_list ? vli + 1 : 0;
      vbase = reinterpret_cast<const char*>(vpool) + head_of(vli) * (size_t)D * P * 2;
    }
  };

  f32x16 acc[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) acc[m] = f32x16{0};
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = p.scale_log2;
  const int krow = key_perm(l32);

  // The lane's byte offsets of its MFMA operands within a tile are fixed:
  // one per d slice (key rows; the second key half is 32 rows further) and
  // one per 16-key step (value rows; output block m is 32 rows further).
  uint32_t offk[KK], offv[4];
#pragma unroll
  for (int j = 0; j < KK; ++j)
    offk[j] = (uint32_t)(krow * L::kRowK + (((2 * j + half) ^ swz_k<D>(krow)) << 4));
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    offv[ks] = (uint32_t)(l32 * L::kRowV + (((2 * ks + half) ^ swz_v(l32)) << 4));
  auto k_tile = [&](int t) { return smem + (t & 3) * L::kKTile; };
  auto v_tile = [&](int t) { return smem + L::kVBase + ((t + 4) & 3) * L::kVTile; };

  f32x16 s[2];
  int tcs = kt;  // tile within its page of the next value phase

  // X(t): the scores of tile t, S^T = K(t) Q^T (two chains, key halves 0 and
  // 1), key fragments read kAheadX MFMAs ahead.
  auto score_phase = [&](int t) {
    constexpr int N = 2 * KK, kAheadX = N < 8 ? N : 8;
    const uint8_t* kt_l = k_tile(t);
    u32x4 f[kAheadX];
#pragma unroll
    for (int i = 0; i < kAheadX; ++i) f[i] = ld_lds16(kt_l + offk[i >> 1] + (i & 1) * 32 * L::kRowK);
    s[0] = f32x16{0};
    s[1] = f32x16{0};
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const u32x4 a = f[i % kAheadX];
      const int n = i + kAheadX;
      if (n < N) f[i % kAheadX] = ld_lds16(kt_l + offk[n >> 1] + (n & 1) * 32 * L::kRowK);
      s[i & 1] = mfma32(a, qf[i >> 1], s[i & 1]);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kAheadX, 0);
#pragma unroll
    for (int i = 0; i < N - kAheadX; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAheadX, 0);
  };

  // Y(t): softmax of the scores of tile t and the value product O^T +=
  // V(t)^T P(t)^T. Each 16-key group's four value MFMAs (one per 32-row
  // output block) are issued as soon as its P fragment is packed, so they
  // run under the exponentials of the next group; value fragments (u = 4 ks
  // + m) are read eight ahead.
  auto value_phase = [&](int t) {
    const uint8_t* vt_l = v_tile(t);
    constexpr int NV = 4 * NM, kAheadV = NV < 8 ? NV : 8;
    auto vop = [&](int u) { return ld_lds16(vt_l + offv[u / NM] + (u % NM) * 32 * L::kRowV); };
    u32x4 f[kAheadV];
#pragma unroll
    for (int u = 0; u < kAheadV; ++u) f[u] = vop(u);
    const int nv = min(kBN, P - tcs * kBN);
    if (nv < kBN) {
      asm volatile("" ::: "memory");
      const int lo = kSmallP ? 0 : kBN - nv, hi = kSmallP ? nv : kBN;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * h2 + 16 * (r >> 3) + 8 * half + (r & 7);
          if (key < lo || key >= hi) s[h2][r] = -INFINITY;
        }
    }
    if (++tcs == tpp) tcs = 0;
    float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
    for (int r = 2; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[1][r]);
    // Online softmax against a reference max m_run (raw score units) that
    // only moves when some score exceeds it by more than 8 in exp2 units:
    // exponentials stay <= 256 and the final normalisation by the row sum
    // is exact for any reference. The test uses each lane's own 32 scores;
    // only when it fires are the two lane halves of a query combined.
    if (__any(mx * c2 > m_run * c2 + 8.f)) {
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const bool grow = mx * c2 > m_run * c2 + 8.f;
      const float m_new = grow ? mx : m_run;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
      l_run *= alpha;
#pragma unroll
      for (int m = 0; m < NM; ++m) acc[m] *= alpha;
      m_run = m_new;
    }
    const float mc = m_run * c2;
    float rs[4];  // row sums per 16-key group
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      // keys 16 ks + 8 half + 0..7 of the tile: score registers 8 (ks & 1) +
      // 0..7 of key half ks >> 1
      float pv[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) pv[r] = __builtin_amdgcn_exp2f(fmaf(s[ks >> 1][8 * (ks & 1) + r], c2, -mc));
      rs[ks] = ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
      const u32x4 pk = u32x4{pack_bf16(pv[0], pv[1]), pack_bf16(pv[2], pv[3]), pack_bf16(pv[4], pv[5]),
                             pack_bf16(pv[6], pv[7])};
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const int u = ks * NM + m;
        const u32x4 a = f[u % kAheadV];
        if (u + kAheadV < NV) f[u % kAheadV] = vop(u + kAheadV);
        acc[m] = mfma32(a, pk, acc[m]);
      }
    }
    l_run += (rs[0] + rs[1]) + (rs[2] + rs[3]);
  };

  if (ntiles > 0) {
    // prologue: K(0), V(0), K(1), V(1), K(2), V(2), then all of them and the
    // query fragments (the compiler does not see the copies; the pinned
    // fragments keep it from waiting for its own loads inside the walk)
    issue_k(0);
    issue_v(0);
    issue_k(1);
    issue_v(1);
    issue_k(2);
    issue_v(2);
    wait_vmcnt<0>();
    // Nothing may be left in flight on the LDS/scalar counter either: a
    // scalar load the compiler issued early for the epilogue would make its
    // wait-count pass assume one pending through the walk, and it then waits
    // for all eight operand reads before the first score MFMA of every phase
    // instead of for one.
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) asm volatile("" : "+v"(qf[kk]));
    // Slot j opens with a barrier. Waves 0-3 run X(t) in slot 2t and Y(t) in
    // slot 2t + 1, waves 4-7 X(t) in slot 2t + 1 and Y(t) in slot 2t + 2; so
    // K(t) is read in slots 2t and 2t + 1 and V(t) in slots 2t + 1 and 2t + 2.
    // After the barrier of slot 2t every wave issues its share of K(t+3) into
    // the ring slot of K(t-1), after that of slot 2t + 1 its share of V(t+3)
    // into that of V(t-1); before the barrier of slot 2t it needs K(t) and
    // before that of slot 2t + 1 V(t), with five of its loads issued after
    // either. Both groups make 2 * ntiles + 1 barriers. The barriers are
    // also hard scheduling boundaries: otherwise the compiler moves
    // register-only work (exponentials, MFMAs) across them and the two
    // groups of a SIMD fall back into step.
    static_assert(L::kInstK == L::kInstV, "one wait count for both rings");
    constexpr int kWait = 5 * L::kInstK;
    auto open_slot = [&](bool wait) {
      __builtin_amdgcn_sched_barrier(0);
      if (wait) wait_vmcnt<kWait>();
      lds_barrier();
      __builtin_amdgcn_sched_barrier(0);
    };
    if (first) {
      for (int t = 0; t < ntiles; ++t) {
        open_slot(t > 0);
        issue_k((t + 3) & 3);
        score_phase(t);
        open_slot(true);
        issue_v((t + 3) & 3);
        value_phase(t);
      }
      open_slot(true);
      issue_k((ntiles + 3) & 3);
    } else {
      open_slot(false);
      issue_k(3);
      for (int t = 0; t < ntiles; ++t) {
        open_slot(true);
        issue_v((t + 3) & 3);
        score_phase(t);
        open_slot(true);
        issue_k((t + 4) & 3);
        value_phase(t);
      }
    }
    wait_vmcnt<0>();  // the trailing re-reads
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
  float lse = l_tot > 0.f ? m_run * p.sm_scale + __logf(l_tot) : -INFINITY;
  const int r_first = p.sc.sk_whole ? 0 : range_of(p.sc, item0);
  const int n_pieces = p.sc.sk_whole ? 1 : range_of(p.sc, item0 + n_tiles_item - 1) - r_first + 1;
  if (n_pieces > 1) {
    // piece k of the item is range r_first + k's first segment (slot 0),
    // except for k = 0 when the item starts inside that range (its last
    // segment, slot 1)
    const int slot0 = item0 != range_start(p.sc, r_first) ? 1 : 0;
    auto cell_of = [&](int k) {
      return ((size_t)(r_first + k) * 2 + (k == 0 ? slot0 : 0)) * 8 + wave;
    };
    if (!last_split_merge<D>(p, cell_of, range_id(p.sc) - r_first, n_pieces, ((size_t)b * H + h) * nqt + qtile,
                             tid, acc, inv_l, lse, smem))
      continue;
  }
  finish<D, 512>(p, smem, b, h, q_idx, qf, acc, inv_l, lse, tid);
  }  // segments
}

// fp32 inputs: VALU attention, 64 queries per workgroup, 4 lanes per query.
// Page mode walks the selected pages and then the current pages; list mode
// walks the 64-key tiles its query block keeps (one query block per
// workgroup: query tile qtile / 2, mask bit qtile % 2 of the tile lists).
template <int D, bool kList>
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnParams p) {
  constexpr int T = 32, BM = 64, DP = D / 4;
  __shared__ float ks[T][D + 1];
  __shared__ float vs[T][D + 1];
  __shared__ float qs[BM][D + 1];
  __shared__ int32_t slots[HSA_MAX_LIST];
  const int tid = threadIdx.x, qr = tid >> 2, part = tid & 3;
  const int qtile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = p.H, P = p.P;
  const float* qg = static_cast<const float*>(p.q);
  const float* kg = static_cast<const float*>(p.k);
  const float* vg = static_cast<const float*>(p.v);
  const int q0 = qtile * BM;
  for (int x = tid; x < BM * D; x += 256) {
    const int r = x / D, dd = x % D;
    const int qi = min(q0 + r, p.n_q - 1);
    qs[r][dd] = qg[(((size_t)b * p.n_q + qi) * H + h) * D + dd];
  }
  float acc[DP];
  for (int e = 0; e < DP; ++e) acc[e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  // keys [off0, off0 + nk) of the page at (slot * H + h) = ph, nk <= T
  auto step = [&](size_t ph, int off0, int nk) {
    __syncthreads();
    const float* kp = kg + ph * P * D;
    const float* vp = vg + ph * D * P;
    for (int x = tid; x < T * D; x += 256) {
      const int key = x / D, dd = x % D;
      ks[key][dd] = key < nk ? kp[(size_t)(off0 + key) * D + dd] : 0.f;
    }
    for (int x = tid; x < T * D; x += 256) {
      const int dd = x / T, key = x % T;
      vs[key][dd] = key < nk ? vp[(size_t)dd * P + off0 + key] : 0.f;
    }
    __syncthreads();
    float sc[T];
    float mx = -INFINITY;
    for (int key = 0; key < T; ++key) {
      float s = 0.f;
      for (int e = 0; e < DP; ++e) s = fmaf(qs[qr][part * DP + e], ks[key][part * DP + e], s);
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      s = key < nk ? s * p.sm_scale : -INFINITY;
      sc[key] = s;
      mx = fmaxf(mx, s);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = expf(m_run - m_new);
    l_run *= alpha;
    for (int e = 0; e < DP; ++e) acc[e] *= alpha;
    for (int key = 0; key < nk; ++key) {
      const float pk = expf(sc[key] - m_new);
      l_run += pk;
      for (int e = 0; e < DP; ++e) acc[e] = fmaf(pk, vs[key][part * DP + e], acc[e]);
    }
    m_run = m_new;
  };
  if constexpr (kList) {
    const size_t cell = ((size_t)b * H + h) * p.sc.nqt + qtile / 2;
    const int len = p.blist_len[cell], bit = qtile & 1;
    const int2* lst = p.blist + cell * p.blist_cap;
    for (int u = 0; u < len; ++u) {
      const int2 e = lst[u];
      if (!((e.y >> bit) & 1)) continue;
      const int k0 = (e.y >> 2) * 64, k1 = min(P, k0 + 64);
      for (int off = k0; off < k1; off += T) step((size_t)e.x, off, min(T, k1 - off));
    }
  } else {
    const int32_t* selrow = p.sel + ((size_t)b * H + h) * p.k_max;
    int n_sel = 0;
    while (n_sel < p.k_max) {
      const int e = selrow[n_sel];
      if (e < 0 || e >= p.max_pages) break;
      ++n_sel;
    }
    const int n_list = n_sel + p.n_cur;
    for (int i = tid; i < n_list; i += 256) {
      const int lp = i < n_sel ? selrow[i] : p.cur_first + (i - n_sel);
      slots[i] = clampi(p.page_table[(size_t)b * p.max_pages + lp], 0, p.num_slots - 1);
    }
    __syncthreads();
    for (int li = 0; li < n_list; ++li)
      for (int off = 0; off < P; off += T) step((size_t)slots[li] * H + h, off, min(T, P - off));
  }
  __syncthreads();  // the query rows are complete even if no key was visited
  const int qi = q0 + qr;
  if (qi >= p.n_q) return;
  const float inv_l = l_run > 0.f ? 1.f / l_run : 0.f;
  if (p.mode == ATTN_SPARSE) {
    float* orow = p.o_sp + (((size_t)b * p.n_q + qi) * H + h) * D + part * DP;
    for (int e = 0; e < DP; ++e) orow[e] = acc[e] * inv_l;
    if (p.lse && part == 0)
      p.lse[((size_t)b * H + h) * p.n_q + qi] = l_run > 0.f ? m_run + logf(l_run) : -INFINITY;
    return;
  }
  const size_t gi = ((size_t)b * p.n_q + qi) * H + h;
  // gate weights of element e of this thread's part of the row
  auto sig = [](const float* g, size_t i) { return g ? 1.f / (1.f + expf(-g[i])) : 0.5f; };
  const float wl_h = p.gate_elem ? 0.f : sig(p.g_lin, gi);
  const float wsp_h = p.gate_elem ? 0.f : sig(p.g_sp, gi);
  auto wl = [&](int e) { return p.gate_elem ? sig(p.g_lin, gi * D + part * DP + e) : wl_h; };
  auto wsp = [&](int e) { return p.gate_elem ? sig(p.g_sp, gi * D + part * DP + e) : wsp_h; };
  float* orow = static_cast<float*>(p.o) + gi * D + part * DP;
  if (p.o_lin) {
    // linear branch from another launch (Linformer): gated sum only
    const float* lrow = p.o_lin + gi * D + part * DP;
    for (int e = 0; e < DP; ++e) orow[e] = wl(e) * lrow[e] + wsp(e) * acc[e] * inv_l;
    return;
  }
  const float* st = p.kv_state + ((size_t)b * H + h) * D * D;
  const float* zz = p.k_state + ((size_t)b * H + h) * D;
  float den = 0.f;
  for (int i = 0; i < D; ++i) den = fmaf(phi(qs[qr][i]), zz[i], den);
  for (int e = 0; e < DP; ++e) {
    const int j = part * DP + e;
    float num = 0.f;
    for (int i = 0; i < D; ++i) num = fmaf(phi(qs[qr][i]), st[(size_t)j * D + i], num);
    orow[e] = wl(e) * (num / den) + wsp(e) * acc[e] * inv_l;
  }
}

}  // namespace

// Partials are kept per 32-query wave slot; the widest workgroup pads the
// query count the most.
static size_t partial_cells(int B, int n_q, int n_part) {
  const size_t nq32 = (size_t)((n_q + kWaveQ * kMaxWaves - 1) / (kWaveQ * kMaxWaves)) * kMaxWaves;
  return (size_t)B * n_part * nq32;
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

size_t attention_partial_o_bytes(int B, int d, int n_q, int n_part) {
  return align256(partial_cells(B, n_q, n_part) * kWaveQ * d * 4);
}

size_t attention_partial_lse_bytes(int B, int n_q, int n_part) {
  return align256(partial_cells(B, n_q, n_part) * 64 * 4);
}

size_t attention_partial_bytes(int B, int H, int d, int n_q, int n_part) {
  // one counter per (b, h, query tile) of the narrowest workgroup (128 queries)
  const size_t ctr = align256((size_t)B * H * ((n_q + 127) / 128) * 4);
  return attention_partial_o_bytes(B, d, n_q, n_part) + attention_partial_lse_bytes(B, n_q, n_part) + ctr;
}

namespace {

// One chunk of the schedule: len consecutive items starting at start, all of
// one (head, split) and so of equal cost (in 64-key tiles).
struct Chunk {
  int start, len;
  double cost;
};

// Workgroup w of a launch runs on XCD w % 8, and each XCD hands its
// workgroups, in order, to whichever of its slots (32 CUs x the workgroups a
// CU holds) frees first. Simulates that for the chunks given XCD by XCD
// (list scheduling): chunks are taken largest item first, each goes to the
// XCD where its items can all start earliest. Returns the simulated
// makespan; fills xcd_of.
double deal_chunks(const std::vector<Chunk>& chunks, int kSlotsPerXcd, std::vector<int>& xcd_of) {
  constexpr int kXcd = 8;
  // slot finish times of each XCD, kept sorted ascending
  std::vector<double> slot(kXcd * kSlotsPerXcd, 0.0);
  xcd_of.assign(chunks.size(), 0);
  for (size_t ci = 0; ci < chunks.size(); ++ci) {
    const Chunk& c = chunks[ci];
    const int L = std::min(c.len, kSlotsPerXcd);
    int best = 0;
    for (int x = 1; x < kXcd; ++x)
      if (slot[x * kSlotsPerXcd + L - 1] < slot[best * kSlotsPerXcd + L - 1]) best = x;
    xcd_of[ci] = best;
    double* s = slot.data() + best * kSlotsPerXcd;
    const double unit = c.cost / c.len;
    for (int k = 0; k < c.len; ++k) {  // list-schedule the chunk's items
      const double v = s[0] + unit;
      double* pos = std::upper_bound(s + 1, s + kSlotsPerXcd, v);
      std::copy(s + 1, pos, s);
      pos[-1] = v;
    }
  }
  double makespan = 0.0;
  for (int x = 0; x < kXcd; ++x) makespan = std::max(makespan, slot[x * kSlotsPerXcd + kSlotsPerXcd - 1]);
  return makespan;
}

// Inputs of a schedule, the key of the schedule cache.
struct PlanKey {
  int B, H, d, n_q, P, max_part, split, waves;
  int list_len[HSA_MAX_HEADS];
  bool operator==(const PlanKey& o) const {
    return B == o.B && H == o.H && d == o.d && n_q == o.n_q && P == o.P && max_part == o.max_part &&
           split == o.split && waves == o.waves && std::equal(list_len, list_len + H, o.list_len);
  }
};

bool plan_schedule(AttnParams& p, int H, int d, int n_q, int P, const int* list_len, int max_part,
                   bool split, int waves);
bool plan_stream_k(AttnParams& p, int B, int H, int n_q, int P, const int* list_len, int max_part,
                   bool split);

}  // namespace

bool plan_attention(AttnParams& p, int B, int H, int d, int n_q, int P, const int* list_len,
                    int max_part, bool split, int waves) {
  constexpr int kCache = 8;
  static std::mutex mu;
  static PlanKey keys[kCache];
  static AttnSchedule scheds[kCache];
  static int n_cached = 0, next = 0;
  PlanKey key{B, H, d, n_q, P, max_part, split ? 1 : 0, waves, {}};
  std::copy(list_len, list_len + H, key.list_len);
  {
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < n_cached; ++i)
      if (keys[i] == key) {
        p.sc = scheds[i];
        return true;
      }
  }
  if (waves == 8 ? !plan_stream_k(p, B, H, n_q, P, list_len, max_part, split)
                 : !plan_schedule(p, H, d, n_q, P, list_len, max_part, split, waves))
    return false;
  std::lock_guard<std::mutex> lock(mu);
  keys[next] = key;
  scheds[next] = p.sc;
  next = (next + 1) % kCache;
  n_cached = std::min(n_cached + 1, kCache);
  return true;
}

namespace {

// Stream-K ranges of the page walk. The launch's items (b, h, 256-query
// tile; a head's items all cost its list's tiles) are laid end to end, tile
// by tile, and cut into G equal ranges of consecutive tiles, one workgroup
// each: G = 256 (one per CU) unless the launch has fewer than 16 tiles per
// range or two ranges per item (the partial slots: each range holds at most
// two pieces of cut items, its first and last segments). Items of equal
// length that fill at least 7/8 of the CUs whole (one or more per range)
// are not cut: the partial outputs, merges and second prologues of cut
// items cost more there than the idle CUs. Launches of at least 4 x 256
// items, and launches of at most 256 items whose longest item is at most
// kCutTiles longer than a range, take one whole item per workgroup
// (sk_whole): with many items per
// range, the 32 ranges running on an XCD would each walk a different head
// and share no page in its L2 (30 batched layers of the streaming workload:
// 17.4 against 14.7 ms per chunk), while the dispatcher's own balancing
// leaves a tail of at most one item in four. split = false (fp32, whose
// kernel does not read the schedule) takes one range.
bool plan_stream_k(AttnParams& p, int B, int H, int n_q, int P, const int* list_len, int max_part,
                   bool split) {
  constexpr int kMaxRanges = 256, kMinTiles = 16, kWholeItems = 4 * kMaxRanges, kCutTiles = 4;
  const int nqt = (n_q + 255) / 256, tpp = (P + kBN - 1) / kBN;
  int64_t per_b = 0;
  for (int h = 0; h < H; ++h) {
    p.sc.sk_head_off[h] = (int32_t)per_b;
    per_b += (int64_t)nqt * std::max(1, list_len[h]) * tpp;
  }
  const int64_t T = (int64_t)B * per_b, items = (int64_t)B * H * nqt;
  if (T > INT32_MAX / 2) return false;  // the kernel indexes tiles in 32 bits
  int64_t G = std::max<int64_t>(1, std::min<int64_t>({kMaxRanges, T / kMinTiles, 2 * items}));
  bool equal = true;
  for (int h = 1; h < H; ++h) equal = equal && std::max(1, list_len[h]) == std::max(1, list_len[0]);
  if (equal) {
    const int64_t k = (items + kMaxRanges - 1) / kMaxRanges;  // items per range
    if (items % k == 0 && 8 * (items / k) >= 7 * kMaxRanges) G = items / k;
  }
  // whole items also when the launch holds at most one item per CU and its
  // longest item is at most a few tiles longer than a range: cutting then
  // saves less than the second prologue and the merge of a cut item cost
  // (the Linformer branch over compressed pages: items of 5-19 tiles)
  int max_len = 1;
  for (int h = 0; h < H; ++h) max_len = std::max(max_len, std::max(1, list_len[h]) * tpp);
  const bool whole = split && items <= INT32_MAX &&
                     (items >= kWholeItems || (items <= kMaxRanges && max_len <= T / G + kCutTiles));
  if (whole) G = items;
  if (!split) G = 1;
  // ranges [0, rm) hold q + 1 tiles, the others q
  const int64_t q = T / G, rm = T % G;
  auto range_of = [&](int64_t t) {
    return (int)(t < rm * (q + 1) ? t / (q + 1) : rm + (t - rm * (q + 1)) / q);
  };
  // the most pieces an item of head h is cut into
  int pieces[HSA_MAX_HEADS];
  bool cut = false;
  for (int h = 0; h < H; ++h) {
    pieces[h] = 1;
    const int64_t len = (int64_t)std::max(1, list_len[h]) * tpp;
    for (int b = 0; b < B && !whole; ++b)
      for (int qt = 0; qt < nqt; ++qt) {
        const int64_t t0 = b * per_b + p.sc.sk_head_off[h] + qt * len;
        pieces[h] = std::max(pieces[h], range_of(t0 + len - 1) - range_of(t0) + 1);
      }
    cut = cut || pieces[h] > 1;
  }
  // partial slots: two per range and wave, in units of a batch entry's
  // 32-query wave slots (G <= 2 items keeps this within 4 per head)
  const int nq32 = nqt * 8;
  const int n_part = cut ? (int)((16 * G + (int64_t)B * nq32 - 1) / ((int64_t)B * nq32)) : 0;
  if (n_part > max_part) return false;
  p.sc.nqt = nqt;
  p.sc.nq32 = nq32;
  p.sc.waves = 8;
  p.sc.n_items = H * nqt;
  p.sc.n_order = H;
  for (int h = 0; h < H; ++h) {
    p.sc.head_order[h] = h;
    p.sc.item_off[h] = h * nqt;
    p.sc.n_split[h] = pieces[h];
    p.sc.list_len[h] = list_len[h];
    p.sc.part_base[h] = 0;
  }
  p.sc.item_off[H] = H * nqt;
  p.sc.n_part = n_part;
  p.sc.n_chunks = (int)G;
  p.sc.xcd_items = (int)((G + 7) / 8);
  p.sc.n_chead = cut ? 1 : 0;
  p.sc.sk_g = (int)G;
  p.sc.sk_q = (int)q;
  p.sc.sk_rm = (int)rm;
  p.sc.sk_whole = whole ? 1 : 0;
  p.sc.sk_head_off[H] = (int32_t)per_b;
  return true;
}

bool plan_schedule(AttnParams& p, int H, int d, int n_q, int P, const int* list_len, int max_part,
                   bool split, int waves) {
  const int kBM = kWaveQ * waves;
  const int nqt = (n_q + kBM - 1) / kBM;
  const int slots_per_xcd = 32 * (8 / waves);
  const int tpp = (P + kBN - 1) / kBN;
  // Cost model (unit: one 64-key tile of one item with a full CU, i.e. two
  // 4-wave or one 8-wave workgroup): an item costs its tiles plus a fixed
  // prologue/epilogue; an item of a split head also writes its partial
  // output, and the last split of each query tile reads them all back and
  // merges them.
  constexpr double kOverheadTiles = 3.0, kTileUs = 2.25, kSplitTiles = 1.5;
  // Items of one batch entry are numbered head by head (heads in decreasing
  // split size), split-major, query tile fastest. The chunks of a (head,
  // split) group read the same pages, so each XCD should run few groups;
  // cutting groups into more chunks balances the XCDs better.
  // Returns false when the (head, split) groups alone exceed the chunk table.
  auto build = [&](const int* ns, int per_group, std::vector<int>& order, std::vector<Chunk>& chunks) {
    order.resize(H);
    for (int h = 0; h < H; ++h) order[h] = h;
    auto split_size = [&](int h) { return (list_len[h] + ns[h] - 1) / ns[h]; };
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return split_size(a) > split_size(b); });
    int groups = 0;
    for (int h = 0; h < H; ++h) groups += ns[h];
    // every group has nqt items, cut into ceil(nqt / len_c) chunks; the
    // table holds HSA_MAX_CHUNKS of them
    const int per_group_max = HSA_MAX_CHUNKS / groups;
    chunks.clear();
    if (per_group_max < 1) return false;
    const int len_c = std::max((nqt + per_group_max - 1) / per_group_max,
                               (nqt + per_group - 1) / per_group);
    for (int i = 0, it = 0; i < H; ++i) {
      const int h = order[i], base = list_len[h] / ns[h], rem = list_len[h] % ns[h];
      for (int sp = 0; sp < ns[h]; ++sp, it += nqt) {
        const double c = (base + (sp < rem ? 1 : 0)) * (double)tpp + kOverheadTiles +
                         (ns[h] > 1 ? kSplitTiles : 0.0);
        for (int a = 0; a < nqt; a += len_c) {
          const int len = std::min(len_c, nqt - a);
          chunks.push_back({it + a, len, c * len});
        }
      }
    }
    // largest item cost first (stable: groups stay in item order)
    std::stable_sort(chunks.begin(), chunks.end(),
                     [](const Chunk& a, const Chunk& b) { return a.cost / a.len > b.cost / b.len; });
    return (int)chunks.size() <= HSA_MAX_CHUNKS;
  };
  std::vector<int> order, xcd_of;
  std::vector<Chunk> chunks;
  constexpr double kInfeasible = 1e30;
  auto evaluate = [&](const int* ns, int per_group) -> double {
    int n_part = 0;
    for (int h = 0; h < H; ++h)
      if (ns[h] > 1) n_part += ns[h];
    if (n_part > max_part) return kInfeasible;
    if (!build(ns, per_group, order, chunks)) return kInfeasible;
    return deal_chunks(chunks, slots_per_xcd, xcd_of) * kTileUs * (waves / 4.0);
  };
  // Search. Start with every head whole; then, one key range at a time, split
  // further the heads whose items are the longest, keeping the split counts
  // of the best simulated launch (a split has to win clearly: it costs
  // partial traffic). Each state tries whole (head, split) groups per XCD and
  // groups cut into 2 or 4 chunks (finer cuts balance the XCDs better but
  // make more XCDs fetch the same pages, so they too have to win clearly).
  // The search stops three splits after the last improvement, or once the
  // simulated launch is within 2% of the perfectly balanced one.
  auto best_cut = [&](const int* ns, int& g_out) {
    double b = kInfeasible;
    for (int g : {1, 2, 4}) {
      const double c = evaluate(ns, g) * (g == 1 ? 1.0 : g == 2 ? 1.01 : 1.03);
      if (c < b) {
        b = c;
        g_out = g;
      }
    }
    return b;
  };
  double total_tiles = 0.0;
  for (int h = 0; h < H; ++h) total_tiles += (double)nqt * (list_len[h] * (double)tpp + kOverheadTiles);
  const double bound = total_tiles / (8.0 * slots_per_xcd) * kTileUs * (waves / 4.0);
  int best_ns[HSA_MAX_HEADS], ns[HSA_MAX_HEADS];
  for (int h = 0; h < H; ++h) best_ns[h] = ns[h] = 1;
  int best_g = 1, g = 1;
  double best = best_cut(ns, best_g);
  if (split) {
    int misses = 0;
    while (misses < 3 && best > 1.02 * bound) {
      // the longest items: every head tied at the largest pages per split
      int longest = 0;
      for (int h = 0; h < H; ++h)
        if (ns[h] < list_len[h]) longest = std::max(longest, (list_len[h] + ns[h] - 1) / ns[h]);
      if (longest <= 1) break;
      for (int h = 0; h < H; ++h)
        if (ns[h] < list_len[h] && (list_len[h] + ns[h] - 1) / ns[h] == longest) ++ns[h];
      const double c = best_cut(ns, g);
      if (c < 0.99 * best) {
        best = c;
        best_g = g;
        std::copy(ns, ns + H, best_ns);
        misses = 0;
      } else {
        ++misses;
      }
    }
  }
  // rebuild order, chunks and xcd_of of the choice (the unsplit plan, the
  // first candidate, always fits: at most HSA_MAX_HEADS groups)
  if (evaluate(best_ns, best_g) >= kInfeasible || chunks.size() > (size_t)HSA_MAX_CHUNKS) return false;
  p.sc.nqt = nqt;
  p.sc.nq32 = nqt * waves;
  p.sc.waves = waves;
  p.sc.n_order = H;
  int items = 0, n_part = 0, n_chead = 0;
  for (int i = 0; i < H; ++i) {
    const int h = order[i];
    p.sc.head_order[i] = h;
    p.sc.item_off[i] = items;
    items += best_ns[h] * nqt;
  }
  p.sc.item_off[H] = items;
  p.sc.n_items = items;
  for (int h = 0; h < H; ++h) {
    p.sc.n_split[h] = best_ns[h];
    p.sc.list_len[h] = list_len[h];
    p.sc.part_base[h] = 0;
    if (best_ns[h] > 1) {
      p.sc.part_base[h] = n_part;
      n_part += best_ns[h];
      ++n_chead;
    }
  }
  p.sc.n_part = n_part;
  p.sc.n_chead = n_chead;
  // each XCD runs its chunks in the order they were dealt to it
  int n = 0, widest = 0;
  for (int x = 0; x < 8; ++x) {
    p.sc.xcd_chunk[x] = n;
    int cnt = 0;
    for (size_t ci = 0; ci < chunks.size(); ++ci)
      if (xcd_of[ci] == x) {
        p.sc.chunk_start[n] = chunks[ci].start;
        p.sc.chunk_len[n] = chunks[ci].len;
        cnt += chunks[ci].len;
        ++n;
      }
    widest = std::max(widest, cnt);
  }
  p.sc.xcd_chunk[8] = n;
  p.sc.n_chunks = n;
  p.sc.xcd_items = widest;
  return true;
}

}  // namespace

hipError_t launch_attention(int dtype, int d, int B, const AttnParams& p, hipStream_t s) {
  if (dtype == HSA_DTYPE_BF16) {
    if (p.sc.n_chead > 0) {
      // arrival counters of the split tiles (a fill kernel, not a memset, so
      // that the launch sequence can be captured into a graph)
      const int n = B * p.H * p.sc.nqt;
      zero_counters_kernel<<<(n + 255) / 256, 256, 0, s>>>(p.attn_ctr, n);
    }
    const bool small = p.P < kBN, list = p.blist != nullptr;
    // tile lists (block-sparse mode) are built per 128-query tile and walked
    // by 4-wave workgroups; the page walk takes 8-wave ones, one per range
    if (p.sc.waves != (list ? 4 : 8)) return hipErrorInvalidValue;
    const dim3 grid = list ? dim3(8 * std::max(1, p.sc.xcd_items), B) : dim3(p.sc.sk_g);
    if (d == 128) {
      if (list) {
        if (small) attn_bf16_kernel<128, true, 4><<<grid, 256, 0, s>>>(p);
        else attn_bf16_kernel<128, false, 4><<<grid, 256, 0, s>>>(p);
      } else {
        if (small) attn_pp_kernel<128, true><<<grid, 512, 0, s>>>(p);
        else attn_pp_kernel<128, false><<<grid, 512, 0, s>>>(p);
      }
    } else {
      if (list) {
        if (small) attn_bf16_kernel<64, true, 4><<<grid, 256, 0, s>>>(p);
        else attn_bf16_kernel<64, false, 4><<<grid, 256, 0, s>>>(p);
      } else {
        if (small) attn_pp_kernel<64, true><<<grid, 512, 0, s>>>(p);
        else attn_pp_kernel<64, false><<<grid, 512, 0, s>>>(p);
      }
    }

  } else {
    const dim3 grid((p.n_q + 63) / 64, p.H, B);
    if (p.blist) {
      if (d == 128) attn_f32_kernel<128, true><<<grid, 256, 0, s>>>(p);
      else attn_f32_kernel<64, true><<<grid, 256, 0, s>>>(p);
    } else {
      if (d == 128) attn_f32_kernel<128, false><<<grid, 256, 0, s>>>(p);
      else attn_f32_kernel<64, false><<<grid, 256, 0, s>>>(p);
    }
  }
  return hipGetLastError();
}

}  // namespace hsa

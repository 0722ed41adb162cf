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
// Work decomposition (bf16, d = 128 shown): a workgroup owns 128 queries of
// one head, four waves of 32 queries each, and walks the head's key list in
// tiles of 64 keys, double-buffered in LDS. Each wave computes the transposed
// score tile S^T = K Q^T with 32x32x16 bf16 MFMAs so that a lane holds 32
// scores of a single query: the running max needs one cross-lane exchange per
// tile and the accumulator rescale is one multiply per register. The value
// product is O^T += V^T P^T, reading the d-major value pages directly. Key
// rows are fed to the score MFMA in a permuted order so that the score
// registers of a lane already form the bf16 operand of the value MFMA.
#include <float.h>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

constexpr int kBM = 128;   // queries per workgroup (4 waves x 32)
constexpr int kBN = 64;    // keys per tile

template <int D>
struct AttnLayout {
  static constexpr int kRowK = 2 * D;                  // bytes per key row
  static constexpr int kChunksK = D / 8;               // 16-byte chunks per key row
  static constexpr int kKTile = kBN * kRowK;           // K tile bytes
  static constexpr int kVTile = D * kBN * 2;           // V^T tile bytes
  static constexpr int kKV = 2 * (kKTile + kVTile);    // double buffer
  static constexpr int kLin = 2 * D * D * 2;           // state hi + lo (bf16)
  static constexpr int kBytes = kKV > kLin ? kKV : kLin;
  static constexpr int kRowsPerInstK = 1024 / kRowK;   // K rows per 1-KB load
  static constexpr int kInstK = kKTile / 1024 / 4;     // K loads per wave
  static constexpr int kInstV = kVTile / 1024 / 4;     // V^T loads per wave
};

// Swizzle of 16-byte chunks within an LDS row: 16 consecutive rows read at
// one logical chunk land on distinct bank groups.
template <int D>
__device__ __forceinline__ int swz_k(int row) {
  if constexpr (D == 128) return row & 15;
  else return (row >> 1) & 7;
}
__device__ __forceinline__ int swz_v(int row) { return (row >> 1) & 7; }

// Score-tile row m holds key perm(m): bits 2 and 3 swapped, so that lane l's
// score registers 0..7 are keys 8*(l/32)+0..7 and 8..15 are 16+8*(l/32)+0..7.
__device__ __forceinline__ int key_perm(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

struct PageCursor {
  int li, off;  // list index and offset within the page of the tile's first key
};

__device__ __forceinline__ void locate(const PageCursor& base, int x, int P, int& li, int& off) {
  off = base.off + x;
  li = base.li;
  while (off >= P) { off -= P; ++li; }
}

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(AttnParams p) {
  using L = AttnLayout<D>;
  constexpr int KK = D / 16;   // 16-wide d slices
  constexpr int NM = D / 32;   // 32-wide d blocks of the output
  __shared__ __attribute__((aligned(1024))) uint8_t smem[L::kBytes];
  __shared__ int32_t slots[HSA_MAX_LIST];
  __shared__ float zs[D];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int qtile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = p.H, P = p.P;

  // ---- key list: selected pages (up to the first invalid entry), then current pages
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
  const int n_kv = n_list * P;
  const int ntiles = (n_kv + kBN - 1) / kBN;

  // ---- Q fragment: lane holds query (l%32) of this wave, d = 16kk + 8*half + 0..7
  const uint16_t* qb = static_cast<const uint16_t*>(p.q);
  const int q_idx = qtile * kBM + wave * 32 + l32;
  const int q_ld = min(q_idx, p.n_q - 1);
  u32x4 qf[KK];
  {
    const uint16_t* qrow = qb + (((size_t)b * p.n_q + q_ld) * H + h) * D + 8 * half;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = ld_global16(qrow + 16 * kk);
  }
  __syncthreads();  // slots visible

  const uint16_t* kpool = static_cast<const uint16_t*>(p.k);
  const uint16_t* vpool = static_cast<const uint16_t*>(p.v);
  // buffer b: key tile at smem + b*kKTile, value tile at smem + 2*kKTile + b*kVTile

  auto issue = [&](const PageCursor& cur, int tile, int buf) {
    const int key0 = tile * kBN;
#pragma unroll
    for (int n = 0; n < L::kInstK; ++n) {
      const int blk = wave * L::kInstK + n;
      const int r = blk * L::kRowsPerInstK + lane / L::kChunksK;
      const int c = (lane % L::kChunksK) ^ swz_k<D>(r);
      int li, off;
      locate(cur, r, P, li, off);
      if (key0 + r >= n_kv) { li = n_list - 1; off = P - 1; }
      const uint16_t* src = kpool + (((size_t)slots[li] * H + h) * P + off) * D + 8 * c;
      g2lds16(src, smem + buf * L::kKTile + blk * 1024);
    }
#pragma unroll
    for (int n = 0; n < L::kInstV; ++n) {
      const int blk = wave * L::kInstV + n;
      const int r = blk * 8 + (lane >> 3);
      const int c = (lane & 7) ^ swz_v(r);
      int li, off;
      locate(cur, 8 * c, P, li, off);
      if (key0 + 8 * c >= n_kv) { li = n_list - 1; off = P - 8; }
      const uint16_t* src = vpool + (((size_t)slots[li] * H + h) * D + r) * P + off;
      g2lds16(src, smem + 2 * L::kKTile + buf * L::kVTile + blk * 1024);
    }
  };

  f32x16 acc[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) acc[m] = f32x16{0};
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = p.scale_log2;

  PageCursor cur{0, 0};
  if (ntiles > 0) issue(cur, 0, 0);
  const int krow = key_perm(l32);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    wait_vmcnt<0>();
    __syncthreads();
    PageCursor nxt = cur;
    nxt.off += kBN;
    while (nxt.off >= P) { nxt.off -= P; ++nxt.li; }
    if (tile + 1 < ntiles) issue(nxt, tile + 1, buf ^ 1);

    // S^T = K Q^T for the two 32-key halves of the tile
    f32x16 s[2];
    const uint8_t* kt = smem + buf * L::kKTile;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      s[h2] = f32x16{0};
      const int row = 32 * h2 + krow;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int chunk = 2 * kk + half;
        const u32x4 a = ld_lds16(kt + row * L::kRowK + ((chunk ^ swz_k<D>(row)) << 4));
        s[h2] = mfma32(a, qf[kk], s[h2]);
      }
    }
    // mask the tail of the key list
    if ((tile + 1) * kBN > n_kv) {
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = tile * kBN + 32 * h2 + 16 * (r >> 3) + 8 * half + (r & 7);
          if (key >= n_kv) s[h2][r] = -INFINITY;
        }
    }
    // online softmax (scores in raw units; exp2 with the folded scale)
    float mx = s[0][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[1][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
    const float mc = m_new * c2;
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
        pb[2 * h2 + g] = u32x4{pack_bf16(pv[8 * g + 0], pv[8 * g + 1]), pack_bf16(pv[8 * g + 2], pv[8 * g + 3]),
                               pack_bf16(pv[8 * g + 4], pv[8 * g + 5]), pack_bf16(pv[8 * g + 6], pv[8 * g + 7])};
    }
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int m = 0; m < NM; ++m) acc[m] *= alpha;
    // O^T += V^T P^T
    const uint8_t* vt = smem + 2 * L::kKTile + buf * L::kVTile;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int chunk = 2 * ks + half;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const int row = 32 * m + l32;
        const u32x4 a = ld_lds16(vt + row * 128 + ((chunk ^ swz_v(row)) << 4));
        acc[m] = mfma32(a, pb[ks], acc[m]);
      }
    }
    cur = nxt;
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
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
      if (p.lse && half == 0)
        p.lse[((size_t)b * H + h) * p.n_q + q_idx] =
            l_tot > 0.f ? m_run * p.sm_scale + __logf(l_tot) : -INFINITY;
    }
    return;
  }

  // ---- linear branch: O_lin^T = S^T phi(Q)^T / (phi(Q) . z), state split
  // into bf16 hi + lo parts so the product keeps ~16 bits of the state.
  __syncthreads();  // all waves are done with the key/value tiles
  uint8_t* sh = smem;
  uint8_t* sl = smem + D * D * 2;
  {
    const float* st = p.kv_state + ((size_t)b * H + h) * D * D;
    for (int e = 4 * tid; e < D * D; e += 1024) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(st + e);
      const int j = e / D, i = e % D;
      const int off = j * (2 * D) + (((i >> 3) ^ swz_k<D>(j)) << 4) + (i & 7) * 2;
      const float hx[4] = {x.x, x.y, x.z, x.w};
      float lo[4];
      uint32_t hw[2], lw[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        hw[t] = pack_bf16(hx[2 * t], hx[2 * t + 1]);
        lo[2 * t] = hx[2 * t] - bf16_lo(hw[t]);
        lo[2 * t + 1] = hx[2 * t + 1] - bf16_hi(hw[t]);
        lw[t] = pack_bf16(lo[2 * t], lo[2 * t + 1]);
      }
      *reinterpret_cast<u32x2*>(sh + off) = u32x2{hw[0], hw[1]};
      *reinterpret_cast<u32x2*>(sl + off) = u32x2{lw[0], lw[1]};
    }
    if (tid < D) zs[tid] = p.k_state[((size_t)b * H + h) * D + tid];
  }
  __syncthreads();
  u32x4 fq[KK];
  float den = 0.f;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const uint32_t w[4] = {qf[kk].x, qf[kk].y, qf[kk].z, qf[kk].w};
    uint32_t o4[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      o4[t] = pack_bf16(phi(bf16_lo(w[t])), phi(bf16_hi(w[t])));
      const int d0 = 16 * kk + 8 * half + 2 * t;
      den = fmaf(bf16_lo(o4[t]), zs[d0], den);
      den = fmaf(bf16_hi(o4[t]), zs[d0 + 1], den);
    }
    fq[kk] = u32x4{o4[0], o4[1], o4[2], o4[3]};
  }
  den += __shfl_xor(den, 32);
  const float inv_den = 1.f / den;
  float wl = 0.5f, wsp = 0.5f;
  if (q_ok) {
    const size_t gi = ((size_t)b * p.n_q + q_idx) * H + h;
    if (p.g_lin) wl = 1.f / (1.f + __expf(-p.g_lin[gi]));
    if (p.g_sp) wsp = 1.f / (1.f + __expf(-p.g_sp[gi]));
  }
  const float a_lin = wl * inv_den, a_sp = wsp * inv_l;
  void* orow_v = nullptr;
  if (q_ok) orow_v = static_cast<uint16_t*>(p.o) + (((size_t)b * p.n_q + q_idx) * H + h) * D;
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    f32x16 al = f32x16{0};
    const int row = 32 * m + l32;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int off = row * (2 * D) + (((2 * kk + half) ^ swz_k<D>(row)) << 4);
      al = mfma32(ld_lds16(sh + off), fq[kk], al);
      al = mfma32(ld_lds16(sl + off), fq[kk], al);
    }
    if (q_ok) {
      uint16_t* orow = static_cast<uint16_t*>(orow_v);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * m + 8 * g + 4 * half;
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = a_lin * al[4 * g + t] + a_sp * acc[m][4 * g + t];
        *reinterpret_cast<u32x2*>(orow + d0) = u32x2{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
      }
    }
  }
}

// fp32 inputs: VALU attention, 64 queries per workgroup, 4 lanes per query.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnParams p) {
  constexpr int T = 32, BM = 64, DP = D / 4;
  __shared__ float ks[T][D + 1];
  __shared__ float vs[T][D + 1];
  __shared__ float qs[BM][D + 1];
  __shared__ int32_t slots[HSA_MAX_LIST];
  const int tid = threadIdx.x, qr = tid >> 2, part = tid & 3;
  const int qtile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int H = p.H, P = p.P;
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
  const int n_kv = n_list * P;
  const float* qg = static_cast<const float*>(p.q);
  const float* kg = static_cast<const float*>(p.k);
  const float* vg = static_cast<const float*>(p.v);
  const int q0 = qtile * BM;
  for (int x = tid; x < BM * D; x += 256) {
    const int r = x / D, dd = x % D;
    const int qi = min(q0 + r, p.n_q - 1);
    qs[r][dd] = qg[(((size_t)b * p.n_q + qi) * H + h) * D + dd];
  }
  __syncthreads();
  float acc[DP];
  for (int e = 0; e < DP; ++e) acc[e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  for (int k0 = 0; k0 < n_kv; k0 += T) {
    const int nk = min(T, n_kv - k0);
    __syncthreads();
    for (int x = tid; x < T * D; x += 256) {
      const int key = x / D, dd = x % D;
      float kv = 0.f;
      if (key < nk) {
        const int j = k0 + key, li = j / P, off = j % P;
        kv = kg[(((size_t)slots[li] * H + h) * P + off) * D + dd];
      }
      ks[key][dd] = kv;
    }
    for (int x = tid; x < T * D; x += 256) {
      const int dd = x / T, key = x % T;
      float vv = 0.f;
      if (key < nk) {
        const int j = k0 + key, li = j / P, off = j % P;
        vv = vg[(((size_t)slots[li] * H + h) * D + dd) * P + off];
      }
      vs[key][dd] = vv;
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
  }
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
  const float* st = p.kv_state + ((size_t)b * H + h) * D * D;
  const float* zz = p.k_state + ((size_t)b * H + h) * D;
  float den = 0.f;
  for (int i = 0; i < D; ++i) den = fmaf(phi(qs[qr][i]), zz[i], den);
  const size_t gi = ((size_t)b * p.n_q + qi) * H + h;
  const float wl = p.g_lin ? 1.f / (1.f + expf(-p.g_lin[gi])) : 0.5f;
  const float wsp = p.g_sp ? 1.f / (1.f + expf(-p.g_sp[gi])) : 0.5f;
  float* orow = static_cast<float*>(p.o) + gi * D + part * DP;
  for (int e = 0; e < DP; ++e) {
    const int j = part * DP + e;
    float num = 0.f;
    for (int i = 0; i < D; ++i) num = fmaf(phi(qs[qr][i]), st[(size_t)j * D + i], num);
    orow[e] = wl * (num / den) + wsp * acc[e] * inv_l;
  }
}

}  // namespace

hipError_t launch_attention(int dtype, int d, int B, const AttnParams& p, hipStream_t s) {
  if (dtype == HSA_DTYPE_BF16) {
    const dim3 grid((p.n_q + kBM - 1) / kBM, p.H, B);
    if (d == 128) attn_bf16_kernel<128><<<grid, 256, 0, s>>>(p);
    else attn_bf16_kernel<64><<<grid, 256, 0, s>>>(p);
  } else {
    const dim3 grid((p.n_q + 63) / 64, p.H, B);
    if (d == 128) attn_f32_kernel<128><<<grid, 256, 0, s>>>(p);
    else attn_f32_kernel<64><<<grid, 256, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace hsa

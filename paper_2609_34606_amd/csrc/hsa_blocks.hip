// Head-adaptive block selection of the sparse branch (Sec. 3.3 "Sparse
// branch" and "Head-level sparsity adaptation"; the appendix on the sparse
// branch gives the pooled map, the coverage rule and the Gini coefficient).
//
// For one head, the active pages (selected history pages, then the current
// pages) are cut into key blocks: kBlockHist tokens in a history page,
// kBlockCur tokens in a current page. The query chunk is cut into blocks of
// kBlockQ queries. With qbar_i and kbar_j the block means,
//   p_i = softmax_j(scale * qbar_i . kbar_j)                (pooled map)
//   G   = mean_i (1/N) sum_m (N - 2m + 1) p_i,(m)           (Gini, weights sorted descending)
//   tau = tau_min + G (tau_max - tau_min)
// and query block i keeps the shortest prefix of its blocks in descending
// weight (equal weights: lower block id first) whose running weight reaches
// tau (all blocks if rounding keeps it below, and all blocks for tau >= 1).
// Everything is fp64.
//
// Three launches:
//   1. block_kmean: one workgroup per (b, h, key block) sums the block's keys
//      (exact in fp64 for bf16 keys) and writes the mean, d-major.
//   2. pooled_rows: one workgroup per (b, h, 4 query blocks) scores the
//      blocks (a thread per key block), then each of four waves takes one
//      query block: softmax, a bitonic sort (in registers up to 1024 blocks,
//      else in LDS), the Gini term and the running weight in sorted order.
//   3. block_lists: one workgroup per (b, h, 128-query tile) forms the
//      threshold from every query block's Gini term (same order in every
//      workgroup), cuts the two prefixes of its query blocks and writes the
//      tile list the attention kernel walks: the union of both kept sets in
//      list order, every 64-key tile with a bit per query block.
#include <float.h>
#include <limits.h>

#include <algorithm>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

// threads of a pooled_rows workgroup: one key block per thread in the score
// loop (up to 512 blocks), then one wave per query block
constexpr int kRowsThreads = 512;

template <typename T>
__device__ __forceinline__ void load8(const T* p, double (&x)[8]);

template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, double (&x)[8]) {
  const u32x4 v = ld_global16(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = (double)bf16_lo(w[e]);
    x[2 * e + 1] = (double)bf16_hi(w[e]);
  }
}

template <>
__device__ __forceinline__ void load8<float>(const float* p, double (&x)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// Orders LDS accesses of one wave: every access before it is complete and
// visible to the wave's other lanes before any access after it.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmax(v, __shfl_xor(v, m));
  return v;
}

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m));
  return v;
}

// Key blocks of one head's list.
struct ListGeom {
  int n_sel;       // valid entries of the selection row
  int nbh, nbc;    // blocks per history / current page
  int n_hist_blk;  // blocks of the history pages
  int n_blk;       // all blocks
};

__device__ __forceinline__ ListGeom list_geom(const BlockSelParams& p, const int32_t* selrow) {
  ListGeom g;
  int n = 0;
  while (n < p.k_max) {
    const int e = selrow[n];
    if (e < 0 || e >= p.max_pages) break;
    ++n;
  }
  g.n_sel = n;
  g.nbh = (p.P + kBlockHist - 1) / kBlockHist;
  g.nbc = (p.P + kBlockCur - 1) / kBlockCur;
  g.n_hist_blk = n * g.nbh;
  g.n_blk = g.n_hist_blk + p.n_cur * g.nbc;
  return g;
}

// Block j of the list: list position, first key in the page, key count.
__device__ __forceinline__ void block_of(const ListGeom& g, int P, int j, int& li, int& k0, int& nk) {
  if (j < g.n_hist_blk) {
    li = j / g.nbh;
    k0 = (j % g.nbh) * kBlockHist;
    nk = min(kBlockHist, P - k0);
  } else {
    j -= g.n_hist_blk;
    li = g.n_sel + j / g.nbc;
    k0 = (j % g.nbc) * kBlockCur;
    nk = min(kBlockCur, P - k0);
  }
}

__device__ __forceinline__ int slot_of(const BlockSelParams& p, const int32_t* selrow,
                                       const ListGeom& g, int b, int li) {
  const int lp = li < g.n_sel ? selrow[li] : p.cur_first + (li - g.n_sel);
  return clampi(p.page_table[(size_t)b * p.max_pages + lp], 0, p.num_slots - 1);
}

// ---------------------------------------------------------------- 1. block means
template <typename T, int D>
__global__ __launch_bounds__(256) void block_kmean_kernel(BlockSelParams p) {
  constexpr int TPR = D / 8;       // threads per key row (8 values each)
  constexpr int RG = 256 / TPR;    // row groups
  __shared__ double part[RG][D];
  const int j = blockIdx.x, h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int32_t* selrow = p.sel + ((size_t)b * p.H + h) * p.k_max;
  const ListGeom g = list_geom(p, selrow);
  if (j >= g.n_blk) return;
  int li, k0, nk;
  block_of(g, p.P, j, li, k0, nk);
  const int slot = slot_of(p, selrow, g, b, li);
  const T* kp = static_cast<const T*>(p.k) + (((size_t)slot * p.H + h) * p.P + k0) * D;
  const int c8 = tid % TPR, rg = tid / TPR;
  double s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll 4
  for (int r = rg; r < nk; r += RG) {
    double x[8];
    load8<T>(kp + (size_t)r * D + c8 * 8, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] += x[e];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[rg][c8 * 8 + e] = s[e];
  __syncthreads();
  if (tid < D) {
    double t = 0.0;
    for (int q = 0; q < RG; ++q) t += part[q][tid];
    p.kbar_t[(((size_t)b * p.H + h) * D + tid) * p.n_blk_max + j] = t / (double)nk;
  }
}

// One wave sorts n_pad (weight, id) pairs in LDS into the order (weight
// descending, id ascending) with a bitonic network. In each stage a lane
// handles pairs lane + 64c; all of its pairs are read before any is written,
// so the reads of a stage are in flight together (reads after a write to the
// same array would otherwise wait for it). PPL bounds the pairs per lane and
// stage held in registers at once.
template <int PPL>
__device__ void bitonic_sort_wave(double* rp, int32_t* ri, int n_pad, int lane) {
  const int half = n_pad >> 1;
  for (int k = 2; k <= n_pad; k <<= 1) {
    for (int jj = k >> 1; jj > 0; jj >>= 1) {
      for (int x0 = 0; x0 < half; x0 += 64 * PPL) {
        double pa[PPL], pb[PPL];
        int ia[PPL], ib[PPL], ii[PPL];
#pragma unroll
        for (int c = 0; c < PPL; ++c) {
          const int x = x0 + lane + 64 * c;
          ii[c] = ((x & ~(jj - 1)) << 1) | (x & (jj - 1));
          if (x < half) {
            pa[c] = rp[ii[c]];
            pb[c] = rp[ii[c] + jj];
            ia[c] = ri[ii[c]];
            ib[c] = ri[ii[c] + jj];
          }
        }
#pragma unroll
        for (int c = 0; c < PPL; ++c) {
          const int x = x0 + lane + 64 * c;
          if (x < half) {
            const bool a_first = pa[c] > pb[c] || (pa[c] == pb[c] && ia[c] < ib[c]);
            if (a_first != ((ii[c] & k) == 0)) {
              rp[ii[c]] = pb[c];
              rp[ii[c] + jj] = pa[c];
              ri[ii[c]] = ib[c];
              ri[ii[c] + jj] = ia[c];
            }
          }
        }
      }
      wave_sync();
    }
  }
}

// The same order for n_pad = 64 E <= 1024 entries, sorted in registers: lane
// l holds entries l E .. l E + E - 1, so compare-exchanges at distances below
// E stay inside a lane and the others pair lane l with lane l ^ (distance / E)
// through cross-lane shuffles (no LDS round trip and wave barrier per stage).
template <int E>
__device__ void bitonic_sort_regs(double* rp, int32_t* ri, int n_pad, int lane) {
  double w[E];
  int id[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    w[e] = rp[lane * E + e];
    id[e] = ri[lane * E + e];
  }
  for (int k = 2; k <= n_pad; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j >= E) {
        const int m = j / E;
        const bool lower = (lane & m) == 0;  // this lane holds the lower position of each pair
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const double tw = __shfl_xor(w[e], m);
          const int ti = __shfl_xor(id[e], m);
          // selects, not branches: every lane takes the same path
          const bool mine_first = (w[e] > tw) | ((w[e] == tw) & (id[e] < ti));
          const bool desc = ((lane * E + e) & k) == 0;
          const bool take = (desc != mine_first) == lower;
          w[e] = take ? tw : w[e];
          id[e] = take ? ti : id[e];
        }
      } else {
#pragma unroll
        for (int jj = 1; jj < E; jj <<= 1) {
          if (j != jj) continue;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            if (e & jj) continue;
            const double wa = w[e], wb = w[e + jj];
            const int ia = id[e], ib = id[e + jj];
            const bool a_first = (wa > wb) | ((wa == wb) & (ia < ib));
            const bool sw = a_first != (((lane * E + e) & k) == 0);
            w[e] = sw ? wb : wa;
            w[e + jj] = sw ? wa : wb;
            id[e] = sw ? ib : ia;
            id[e + jj] = sw ? ia : ib;
          }
        }
      }
    }
  }
  wave_sync();
#pragma unroll
  for (int e = 0; e < E; ++e) {
    rp[lane * E + e] = w[e];
    ri[lane * E + e] = id[e];
  }
  wave_sync();
}

// ---------------------------------------------------------------- 2. pooled rows
// p.rpg query blocks per workgroup (1..4, one per wave of the first four;
// fewer for long lists so that the rows fit in LDS).
template <int D>
__global__ __launch_bounds__(kRowsThreads) void pooled_rows_kernel(BlockSelParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t dsm[];
  const int rpg = p.rpg;
  double* qbar = reinterpret_cast<double*>(dsm);                   // [rpg][D]
  double* rowp = qbar + rpg * D;                                   // [rpg][n_pad]
  int32_t* rowi = reinterpret_cast<int32_t*>(rowp + rpg * p.n_pad);  // [rpg][n_pad]
  const int h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qb0 = blockIdx.x * rpg;
  const int32_t* selrow = p.sel + ((size_t)b * p.H + h) * p.k_max;
  const ListGeom g = list_geom(p, selrow);
  const int N = g.n_blk;
  const size_t bh = (size_t)b * p.H + h;

  // query block means from the column sums of its two halves
  const int HD = p.H * D;
  for (int x = tid; x < rpg * D; x += kRowsThreads) {
    const int i = x / D, dd = x % D, qb = qb0 + i;
    double v = 0.0;
    if (qb < p.n_qb) {
      const double* qs = p.ws_qs + (size_t)b * p.qs_split * HD + h * D + dd;
      double sum = qs[(size_t)(2 * qb) * HD];
      if (2 * qb + 1 < p.qs_split) sum += qs[(size_t)(2 * qb + 1) * HD];
      v = sum / (double)min(kBlockQ, p.n_q - qb * kBlockQ);
    }
    qbar[i * D + dd] = v;
  }
  __syncthreads();
  // scaled scores of the key blocks against the group's query blocks (rows
  // past rpg read row 0's mean and are not stored)
  const double* kb = p.kbar_t + bh * D * p.n_blk_max;
  int qi[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) qi[i] = (i < rpg ? i : 0) * D;
  for (int j = tid; j < N; j += kRowsThreads) {
    double a[4] = {0, 0, 0, 0};
    // 32 block-mean loads in flight before their FMAs (the sums keep the
    // order dd = 0, 1, ...)
    for (int d0 = 0; d0 < D; d0 += 32) {
      double kv[32];
#pragma unroll
      for (int u = 0; u < 32; ++u) kv[u] = kb[(size_t)(d0 + u) * p.n_blk_max + j];
#pragma unroll
      for (int u = 0; u < 32; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = fma(qbar[qi[i] + d0 + u], kv[u], a[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i < rpg) rowp[i * p.n_pad + j] = a[i] * p.scale;
  }
  __syncthreads();

  // one query block per wave from here on
  const int qb = qb0 + wave;
  if (wave >= rpg || qb >= p.n_qb) return;
  const size_t row = bh * p.n_qb + qb;
  if (N == 0) {
    if (lane == 0) p.row_g[row] = 0.0;
    if (p.pooled)
      for (int j = lane; j < p.kept_len; j += 64) p.pooled[row * p.kept_len + j] = 0.0;
    return;
  }
  double* rp = rowp + wave * p.n_pad;
  int32_t* ri = rowi + wave * p.n_pad;
  double mx = -INFINITY;
  for (int j = lane; j < N; j += 64) mx = fmax(mx, rp[j]);
  mx = wave_max(mx);
  double z = 0.0;
  for (int j = lane; j < N; j += 64) {
    const double e = exp(rp[j] - mx);
    rp[j] = e;
    z += e;
  }
  z = wave_sum(z);
  for (int j = lane; j < p.n_pad; j += 64) {
    if (j < N) {
      const double pj = rp[j] / z;
      rp[j] = pj;
      ri[j] = j;
    } else {
      rp[j] = -1.0;  // padding sorts after every weight
      ri[j] = INT_MAX;
    }
  }
  if (p.pooled)
    for (int j = lane; j < p.kept_len; j += 64) p.pooled[row * p.kept_len + j] = j < N ? rp[j] : 0.0;
  wave_sync();
  // sort: weight descending, block id ascending
  switch (p.n_pad) {
    case 64: bitonic_sort_regs<1>(rp, ri, p.n_pad, lane); break;
    case 128: bitonic_sort_regs<2>(rp, ri, p.n_pad, lane); break;
    case 256: bitonic_sort_regs<4>(rp, ri, p.n_pad, lane); break;
    case 512: bitonic_sort_regs<8>(rp, ri, p.n_pad, lane); break;
    case 1024: bitonic_sort_regs<16>(rp, ri, p.n_pad, lane); break;
    default: bitonic_sort_wave<8>(rp, ri, p.n_pad, lane);
  }
  // Gini term: (1/N) sum over sorted positions m = pos + 1 of (N - 2m + 1) p
  double gs = 0.0;
  for (int pos = lane; pos < N; pos += 64) gs += ((double)(N - 2 * pos - 1) / (double)N) * rp[pos];
  gs = wave_sum(gs);
  if (lane == 0) p.row_g[row] = gs;
  // running weight in sorted order: each lane a contiguous run, then a scan
  // of the run totals across the wave
  const int E = p.n_pad / 64;
  const int r0 = lane * E;
  double tot = 0.0;
  for (int r = 0; r < E; ++r)
    if (r0 + r < N) tot += rp[r0 + r];
  double incl = tot;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  double run = __shfl_up(incl, 1);
  if (lane == 0) run = 0.0;
  double* rc = p.row_c + row * p.n_blk_max;
  int32_t* rix = p.row_i + row * p.n_blk_max;
  for (int r = 0; r < E; ++r) {
    const int pos = r0 + r;
    if (pos < N) {
      run += rp[pos];
      rc[pos] = run;
      rix[pos] = ri[pos];
    }
  }
}

// ---------------------------------------------------------------- 3. tile lists
__global__ __launch_bounds__(256) void block_lists_kernel(BlockSelParams p) {
  __shared__ uint8_t fa[HSA_MAX_BLOCKS], fb[HSA_MAX_BLOCKS];
  __shared__ int wsum[4];
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int32_t* selrow = p.sel + ((size_t)b * p.H + h) * p.k_max;
  const ListGeom g = list_geom(p, selrow);
  const int N = g.n_blk;
  const size_t bh = (size_t)b * p.H + h;
  // threshold of the head: every workgroup sums the Gini terms in the same order
  double gs = 0.0;
  for (int i = lane; i < p.n_qb; i += 64) gs += p.row_g[bh * p.n_qb + i];
  gs = wave_sum(gs);
  const double G = gs / (double)p.n_qb;
  const double tau = p.tau_min + G * (p.tau_max - p.tau_min);
  if (qt == 0 && tid == 0) {
    if (p.gini) p.gini[bh] = G;
    if (p.tau) p.tau[bh] = tau;
  }
  for (int j = tid; j < N; j += 256) fa[j] = fb[j] = 0;
  __syncthreads();
  // kept prefixes of query blocks 2qt (wave 0) and 2qt + 1 (wave 1)
  if (wave < 2) {
    const int qb = 2 * qt + wave;
    if (qb < p.n_qb) {
      const size_t row = bh * p.n_qb + qb;
      const double* rc = p.row_c + row * p.n_blk_max;
      const int32_t* rix = p.row_i + row * p.n_blk_max;
      int first = N;
      for (int m = lane; m < N; m += 64)
        if (rc[m] >= tau) {
          first = m;
          break;
        }
      first = wave_min(first);
      // tau >= 1 is the whole mass: every block, whatever the rounding
      const int k = (first < N && tau < 1.0) ? first + 1 : N;
      uint8_t* f = wave == 0 ? fa : fb;
      for (int m = lane; m < k; m += 64) f[rix[m]] = 1;
      if (p.n_kept && lane == 0) p.n_kept[row] = k;
      if (p.kept)
        for (int m = lane; m < p.kept_len; m += 64) p.kept[row * p.kept_len + m] = m < k ? rix[m] : -1;
    }
  }
  __syncthreads();
  // tile list: kept blocks of either query block in list order, each block's
  // 64-key tiles with the mask of the query blocks that keep it
  const int per = (N + 255) / 256;
  const int j0 = min(N, tid * per), j1 = min(N, j0 + per);
  int cnt = 0;
  for (int j = j0; j < j1; ++j)
    if (fa[j] | fb[j]) {
      int li, k0, nk;
      block_of(g, p.P, j, li, k0, nk);
      cnt += (nk + 63) / 64;
    }
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int pos = incl - cnt;
  for (int w = 0; w < wave; ++w) pos += wsum[w];
  const size_t cell = bh * p.n_qt + qt;
  int2* out = p.blist + cell * p.blist_cap;
  for (int j = j0; j < j1; ++j) {
    const int mask = fa[j] | (fb[j] << 1);
    if (!mask) continue;
    int li, k0, nk;
    block_of(g, p.P, j, li, k0, nk);
    const int ph = slot_of(p, selrow, g, b, li) * p.H + h;
    for (int t = k0 / 64; t < (k0 + nk + 63) / 64; ++t) out[pos++] = make_int2(ph, (t << 2) | mask);
  }
  if (tid == 255) p.blist_len[cell] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
}

}  // namespace

size_t block_rows_lds_bytes(int d, int n_pad, int rpg) {
  return (size_t)rpg * d * 8 + (size_t)rpg * n_pad * 12;
}

hipError_t launch_block_select(int dtype, int d, int B, const BlockSelParams& p, hipStream_t s) {
  const dim3 g1(std::max(1, p.n_blk_max), p.H, B);
  if (dtype == HSA_DTYPE_BF16) {
    if (d == 128) block_kmean_kernel<uint16_t, 128><<<g1, 256, 0, s>>>(p);
    else block_kmean_kernel<uint16_t, 64><<<g1, 256, 0, s>>>(p);
  } else {
    if (d == 128) block_kmean_kernel<float, 128><<<g1, 256, 0, s>>>(p);
    else block_kmean_kernel<float, 64><<<g1, 256, 0, s>>>(p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 g2((p.n_qb + p.rpg - 1) / p.rpg, p.H, B);
  const size_t lds = block_rows_lds_bytes(d, p.n_pad, p.rpg);
  if (d == 128) pooled_rows_kernel<128><<<g2, kRowsThreads, lds, s>>>(p);
  else pooled_rows_kernel<64><<<g2, kRowsThreads, lds, s>>>(p);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 g3(p.n_qt, p.H, B);
  block_lists_kernel<<<g3, 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace hsa

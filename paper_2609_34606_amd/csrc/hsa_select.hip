// Stage-2 page-level retrieval (Sec. 3.2): score every history page of a
// head by qbar . kbar / sqrt(d) and keep the head's top-k_h pages.
//
// Two launches. The first reduces the query chunk to per-split fp64 column
// sums (the chunk is 14 MB at 4680 x 12 x 128 bf16, so it is read by many
// workgroups). The second runs one workgroup per (batch, head): it finishes
// the mean query in a fixed order, scores the candidates in fp64 and takes
// the top k_h by ranking every candidate in the (score desc, index asc)
// order (repeated block-wide arg-max for very long lists), so equal scores
// keep the older page.
#include <float.h>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&x)[8]);

template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float (&x)[8]) {
  const u32x4 v = ld_global16(p);
  x[0] = bf16_lo(v.x); x[1] = bf16_hi(v.x); x[2] = bf16_lo(v.y); x[3] = bf16_hi(v.y);
  x[4] = bf16_lo(v.z); x[5] = bf16_hi(v.z); x[6] = bf16_lo(v.w); x[7] = bf16_hi(v.w);
}

template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&x)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// Column sums of a block of query rows, fp64: ws_qs[b][split][c]. Rows are
// read sixteen at a time so that the loads are in flight together; the sum
// still runs over the rows in increasing order.
template <typename T>
__global__ __launch_bounds__(256) void qsum_kernel(QsumParams p) {
  const int b = blockIdx.y, split = blockIdx.x;
  const int r0 = split * p.rows_per_split;
  const int r1 = min(p.n_q, r0 + p.rows_per_split);
  const T* q = static_cast<const T*>(p.q) + (size_t)b * p.n_q * p.HD;
  const int nvec = p.HD / 8;
  for (int vc = threadIdx.x; vc < nvec; vc += blockDim.x) {
    double s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int r = r0;
    for (; r + 16 <= r1; r += 16) {
      float x[16][8];
#pragma unroll
      for (int u = 0; u < 16; ++u) load8<T>(q + (size_t)(r + u) * p.HD + vc * 8, x[u]);
#pragma unroll
      for (int u = 0; u < 16; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] += (double)x[u][e];
    }
    for (; r < r1; ++r) {
      float x[8];
      load8<T>(q + (size_t)r * p.HD + vc * 8, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += (double)x[e];
    }
    double* out = p.ws_qs + ((size_t)b * p.n_split + split) * p.HD + vc * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = s[e];
  }
}

struct Best {
  double s;
  int i;
};

// (score desc, index asc) order: true if a ranks before b.
__device__ __forceinline__ bool before(const Best& a, const Best& b) {
  return a.s > b.s || (a.s == b.s && a.i < b.i);
}

__device__ __forceinline__ Best shfl_xor_best(Best v, int m) {
  Best o;
  o.s = __shfl_xor(v.s, m);
  o.i = __shfl_xor(v.i, m);
  return o;
}

// One 1024-thread workgroup per (batch, head).
constexpr int kSelThreads = 1024;

template <int D>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p) {
  constexpr int NT = kSelThreads, NW = NT / 64;
  constexpr int DS = D / 16;       // d values per lane when 16 lanes share a candidate
  constexpr int NPART = NT / D;    // threads per column of the mean query
  constexpr int SLOTS = NT / 16;   // candidates scored at once
  constexpr int U = 4;             // candidates per slot with loads in flight together
  __shared__ double qparts[NPART][D];
  __shared__ double qbar[D];
  __shared__ double score[HSA_MAX_CAND];
  __shared__ uint8_t taken[HSA_MAX_CAND];
  __shared__ Best wbest[NW];
  const int bh = blockIdx.x, b = bh / p.H, h = bh % p.H;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // mean query of head h: NPART threads per column each sum a contiguous
  // range of the splits (in order), then the parts are added in order
  {
    const int col = tid % D, part = tid / D;
    const int per = (p.n_split + NPART - 1) / NPART;
    const int k0 = min(p.n_split, part * per), k1 = min(p.n_split, k0 + per);
    const double* src = p.ws_qs + (size_t)b * p.n_split * (p.H * D) + h * D + col;
    double sacc = 0.0;
    int k = k0;
    for (; k + 8 <= k1; k += 8) {
      double x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = src[(size_t)(k + u) * (p.H * D)];
#pragma unroll
      for (int u = 0; u < 8; ++u) sacc += x[u];
    }
    for (; k < k1; ++k) sacc += src[(size_t)k * (p.H * D)];
    qparts[part][col] = sacc;
    __syncthreads();
    if (tid < D) {
      double t = 0.0;
      for (int q = 0; q < NPART; ++q) t += qparts[q][tid];
      qbar[tid] = t / (double)p.n_q;
    }
    __syncthreads();
  }

  // candidates: logical pages [lo, lo + n_c)
  const int lo = p.cand_range ? clampi(p.cand_range[2 * b], 0, p.n_cand) : 0;
  const int n_c = p.cand_range ? clampi(p.cand_range[2 * b + 1], lo, p.n_cand) - lo : p.n_cand;
  // scores: 16 lanes per candidate, DS consecutive dims each, reduced in a
  // fixed butterfly order; U candidates per lane group have their loads in
  // flight together
  const double* km = p.page_kmean + ((size_t)bh * p.max_pages + lo) * D;
  const int sub = tid & 15;
  double qv[DS];
#pragma unroll
  for (int e = 0; e < DS; ++e) qv[e] = qbar[sub * DS + e];
  const double rsd = sqrt((double)D);
  for (int c0 = 0; c0 < n_c; c0 += SLOTS * U) {
    double part[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * SLOTS + (tid >> 4);
      part[u] = 0.0;
      if (c < n_c) {
        const double* kr = km + (size_t)c * D + sub * DS;
#pragma unroll
        for (int e = 0; e < DS; ++e) part[u] = fma(qv[e], kr[e], part[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      double v = part[u];
      v += __shfl_xor(v, 8);
      v += __shfl_xor(v, 4);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 1);
      const int c = c0 + u * SLOTS + (tid >> 4);
      if (sub == 0 && c < n_c) {
        score[c] = v / rsd;
        taken[c] = 0;
      }
    }
  }
  __syncthreads();

  const int k_eff = min(p.k_h[h], n_c);
  int32_t* sel = p.sel + (size_t)bh * p.k_max;
  double* sc = p.sel_score ? p.sel_score + (size_t)bh * p.k_max : nullptr;
  for (int r = k_eff + tid; r < p.k_max; r += NT) {
    sel[r] = -1;
    if (sc) sc[r] = 0.0;
  }
  if (k_eff == 0) return;
  if (n_c <= 2048) {
    // rank of each candidate in the (score desc, index asc) order, counted by
    // G lanes per candidate (each a strided share of the others) and summed
    // across them; ranks are a permutation for comparable scores (rows start
    // at -1 in case a NaN score breaks that)
    for (int r = tid; r < k_eff; r += NT) sel[r] = -1;
    __syncthreads();
    int G = 16;
    while (G > 1 && G * n_c > NT) G >>= 1;
    const int q = tid & (G - 1);
    for (int c = tid / G; c - tid / G < n_c; c += NT / G) {  // uniform trip count per lane group
      const bool mine = c < n_c;
      const Best me{mine ? score[c] : 0.0, c};
      int rank = 0;
      if (mine)
        for (int o = q; o < n_c; o += G) rank += before(Best{score[o], o}, me) ? 1 : 0;
      for (int m = 1; m < G; m <<= 1) rank += __shfl_xor(rank, m);
      if (mine && q == 0 && rank < k_eff) {
        sel[rank] = lo + c;
        if (sc) sc[rank] = me.s;
      }
    }
    return;
  }
  // long candidate lists: k_eff rounds of block-wide arg-max
  for (int r = 0; r < k_eff; ++r) {
    Best best{-DBL_MAX, INT32_MAX};
    bool have = false;
    for (int c = tid; c < n_c; c += NT) {
      if (taken[c]) continue;
      const Best cand{score[c], c};
      if (!have || before(cand, best)) { best = cand; have = true; }
    }
    if (!have) best = Best{-DBL_MAX, INT32_MAX};
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const Best o = shfl_xor_best(best, m);
      if (before(o, best)) best = o;
    }
    if (lane == 0) wbest[wave] = best;
    __syncthreads();
    if (tid == 0) {
      Best bb = wbest[0];
      for (int w = 1; w < NW; ++w)
        if (wbest[w].i < n_c && (bb.i >= n_c || before(wbest[w], bb))) bb = wbest[w];
      // a NaN score can leave no comparable candidate: pad instead of indexing
      const bool ok = bb.i >= 0 && bb.i < n_c;
      if (ok) taken[bb.i] = 1;
      sel[r] = ok ? lo + bb.i : -1;
      if (sc) sc[r] = ok ? bb.s : 0.0;
    }
    __syncthreads();
  }
}

// Stage-1 prompt-level retrieval (Sec. 3.2): one workgroup of 16 waves per
// batch entry. Each wave takes every sixteenth chunk: fp64 dot product and
// norm over the embedding dimension (each lane keeps eight partial sums
// over its elements, added in a fixed pairwise order, then a fixed butterfly
// across the wave), cosine = dot / (|p| |c|), 0 for a zero norm; then the
// top-1 by (cosine desc, index asc) over the workgroup.
constexpr int kChunkWaves = 16;

// Per-lane partial sums of a.b and a.a over E elements: a lane reads VW
// consecutive floats per access (VW = 4: 16-byte loads) and issues U accesses
// of each array per round before using them (the pass is latency-bound: one
// workgroup streams every chunk embedding of its batch entry); the products
// of a round go to eight fp64 partials in a fixed order.
template <int VW>
__device__ __forceinline__ void dot_norm(const float* a, const float* bv, int E, int lane,
                                         double (&dot)[8], double (&na)[8]) {
  constexpr int U = VW == 4 ? 4 : 8;
  const int n = E / VW;
  for (int g0 = lane; g0 < n; g0 += 64 * U) {
    float x[U][VW], y[U][VW];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int g = g0 + 64 * u;
      const bool in = g < n;
      if constexpr (VW == 4) {
        const float4 xa = in ? reinterpret_cast<const float4*>(a)[g] : float4{0.f, 0.f, 0.f, 0.f};
        const float4 ya = in ? reinterpret_cast<const float4*>(bv)[g] : float4{0.f, 0.f, 0.f, 0.f};
        x[u][0] = xa.x; x[u][1] = xa.y; x[u][2] = xa.z; x[u][3] = xa.w;
        y[u][0] = ya.x; y[u][1] = ya.y; y[u][2] = ya.z; y[u][3] = ya.w;
      } else {
        x[u][0] = in ? a[g] : 0.f;
        y[u][0] = in ? bv[g] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        const int k = (u * VW + e) & 7;
        dot[k] = fma((double)x[u][e], (double)y[u][e], dot[k]);
        na[k] = fma((double)x[u][e], (double)x[u][e], na[k]);
      }
  }
}

__global__ __launch_bounds__(64 * kChunkWaves) void chunk_select_kernel(ChunkSelectParams p) {
  __shared__ Best wbest[kChunkWaves];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* pr = p.prompt + (size_t)b * p.E;
  auto wave_sum = [](double v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
  };
  auto lane_sum = [](const double (&a)[8]) {
    return ((a[0] + a[4]) + (a[2] + a[6])) + ((a[1] + a[5]) + (a[3] + a[7]));
  };
  // 16-byte loads when every row starts 16-byte aligned
  const bool vec = (p.E & 3) == 0 && ((uintptr_t)p.prompt & 15) == 0 && ((uintptr_t)p.chunks & 15) == 0;
  auto sums = [&](const float* x, double (&dot)[8], double (&na)[8]) {
#pragma unroll
    for (int k = 0; k < 8; ++k) dot[k] = na[k] = 0.0;
    if (vec) dot_norm<4>(x, pr, p.E, lane, dot, na);
    else dot_norm<1>(x, pr, p.E, lane, dot, na);
  };
  double d8[8], n8[8];
  sums(pr, d8, n8);
  const double pn = wave_sum(lane_sum(n8));
  Best best{-DBL_MAX, INT32_MAX};
  for (int c = wave; c < p.M; c += kChunkWaves) {
    sums(p.chunks + ((size_t)b * p.M + c) * p.E, d8, n8);
    const double dt = wave_sum(lane_sum(d8));
    const double cc = wave_sum(lane_sum(n8));
    const double den = sqrt(cc) * sqrt(pn);
    const Best cand{den > 0.0 ? dt / den : 0.0, c};
    if (best.i == INT32_MAX || before(cand, best)) best = cand;
  }
  if (lane == 0) wbest[wave] = best;
  __syncthreads();
  if (tid == 0) {
    Best bb = wbest[0];
    for (int w = 1; w < kChunkWaves; ++w)
      if (wbest[w].i < p.M && (bb.i >= p.M || before(wbest[w], bb))) bb = wbest[w];
    const int m = bb.i < p.M ? bb.i : 0;
    const int32_t* cf = p.chunk_first + (size_t)b * (p.M + 1);
    const int lo = clampi(cf[m], 0, p.n_cand);
    p.cand_range[2 * b] = lo;
    p.cand_range[2 * b + 1] = clampi(cf[m + 1], lo, p.n_cand);
    if (p.chunk_out) p.chunk_out[b] = m;
    if (p.chunk_score) p.chunk_score[b] = bb.i < p.M ? bb.s : 0.0;
  }
}

}  // namespace

hipError_t launch_chunk_select(int B, const ChunkSelectParams& p, hipStream_t s) {
  chunk_select_kernel<<<B, 64 * kChunkWaves, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_qsum(int dtype, int B, const QsumParams& qp, hipStream_t s) {
  const dim3 g1(qp.n_split, B);
  if (dtype == HSA_DTYPE_BF16) qsum_kernel<uint16_t><<<g1, 256, 0, s>>>(qp);
  else qsum_kernel<float><<<g1, 256, 0, s>>>(qp);
  return hipGetLastError();
}

hipError_t launch_page_select(int dtype, int d, int B, const QsumParams& qp,
                              const SelectParams& sp, hipStream_t s) {
  hipError_t e = launch_qsum(dtype, B, qp, s);
  if (e != hipSuccess) return e;
  const dim3 g2(B * sp.H);
  if (d == 128) select_kernel<128><<<g2, kSelThreads, 0, s>>>(sp);
  else select_kernel<64><<<g2, kSelThreads, 0, s>>>(sp);
  return hipGetLastError();
}

}  // namespace hsa

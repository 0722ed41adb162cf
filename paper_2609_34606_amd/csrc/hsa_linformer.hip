// Linformer compression of pages (Sec. 3.3 "Linear branch"; App. "Linear
// Branch"): with one page as the projection segment (L = P), every page of
// every head is compressed once, when it is written,
//   ck = E_K^T K   (r x d),     cv = (E_V^T V)^T   (d x r, stored d-major),
// with the head's projections given as e_k[h][j][t] = E_K^(h)[t][j]. The
// compressed pages form a KV pool of page size r that the attention kernels
// read like any other pool.
//
// bf16: both products contract over the page's tokens. Value pages are
// stored d-major and the projections rank-major, so their 64-token tiles go
// straight from HBM into LDS (global_load_lds) as MFMA operands; key rows
// come through registers and are written to LDS transposed ([d][token]).
// One workgroup per (page part, head); 32x32x16 bf16 MFMAs with fp32
// accumulation; waves 0-1 own ck's output tiles, waves 2-3 cv's. A page is
// split into parts only when there are too few (page, head) pairs to fill
// the chip; parts write fp32 partials that a second kernel sums in order.
#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

constexpr int kT = 64;          // tokens per LDS tile
constexpr int kRow = kT * 2;    // bytes per LDS row: 64 bf16 tokens

// 16-byte chunk swizzle of 128-byte LDS rows: 16 consecutive rows read at one
// logical chunk land on distinct bank groups.
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 4)) & 7; }

template <int D, int R>
struct CompressSmem {
  uint8_t kt[D * kRow];  // K^T tile [d][64 tokens]
  uint8_t vt[D * kRow];  // V tile [d][64 tokens]
  uint8_t ek[R * kRow];  // E_K^T tile [j][64 tokens]
  uint8_t ev[R * kRow];  // E_V^T tile [j][64 tokens]
};

template <int D, int R, bool kSmallP>
__global__ __launch_bounds__(256) void compress_bf16_kernel(CompressParams p) {
  constexpr int DQ = D / 4, KG = 256 / DQ, KPT = kT / KG;  // key loads: 4 dims x KPT tokens
  constexpr int NMD = D / 32, NMR = R / 32;
  constexpr int NTK = NMR * NMD;       // ck output tiles (cv has as many)
  constexpr int TPW = 2 * NTK / 4;     // output tiles per wave
  constexpr int NV = D / 32;           // 1-KB V loads per wave (8 rows x 128 B each)
  constexpr int NE = R / 32;           // 1-KB loads per wave per projection
  static_assert(KPT == 8 || KPT == 4, "layout");
  __shared__ __attribute__((aligned(16))) CompressSmem<D, R> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int pi = blockIdx.x / p.parts, part = blockIdx.x % p.parts;
  const int page = p.first_page + pi;
  const int slot = clampi(p.page_table[(size_t)b * p.max_pages + page], 0, p.num_slots - 1);
  const size_t hb = (size_t)slot * p.H + h;
  const int P = p.P;
  const int t_beg = part * p.part_len, t_end = min(P, t_beg + p.part_len);

  const uint16_t* kb = static_cast<const uint16_t*>(p.k) + hb * P * D;   // [P][D]
  const uint16_t* vb = static_cast<const uint16_t*>(p.v) + hb * D * P;   // [D][P]
  const uint16_t* ekb = static_cast<const uint16_t*>(p.e_k) + (size_t)h * R * P;  // [R][P]
  const uint16_t* evb = static_cast<const uint16_t*>(p.e_v) + (size_t)h * R * P;
  const int dq = tid % DQ, kg = tid / DQ;

  f32x16 acc[TPW];
#pragma unroll
  for (int q = 0; q < TPW; ++q) acc[q] = f32x16{0};

  for (int t0 = t_beg; t0 < t_end; t0 += kT) {
    const int nv = min(kT, t_end - t0);
    // window of the tile: 64 tokens ending at the page end when fewer remain
    // (rows before the tile's first token are masked), or the whole page
    // when it is shorter than a tile (rows past it are clamped and masked)
    const int ws = kSmallP ? 0 : min(t0, P - kT);
    const int lo = t0 - ws, hi = lo + nv;
    // row-major tiles of 64 tokens: rows r = (wave * n_inst + n) * 8 + lane / 8,
    // source chunk (lane % 8) ^ swz(r) lands at chunk lane % 8 of row r
    auto row_load = [&](const uint16_t* base, int n_inst, uint8_t* dst, int n) {
      const int r = (wave * n_inst + n) * 8 + (lane >> 3);
      int col = 8 * ((lane & 7) ^ swz(r));
      if constexpr (kSmallP) col = min(col, P - 8);
      g2lds16(base + (size_t)r * P + ws + col, dst + (wave * n_inst + n) * 1024);
    };
#pragma unroll
    for (int n = 0; n < NV; ++n) row_load(vb, NV, sm.vt, n);
#pragma unroll
    for (int n = 0; n < NE; ++n) row_load(ekb, NE, sm.ek, n);
#pragma unroll
    for (int n = 0; n < NE; ++n) row_load(evb, NE, sm.ev, n);
    u32x2 kr[KPT];
#pragma unroll
    for (int e = 0; e < KPT; ++e) {
      int row = kg * KPT + e;
      if constexpr (kSmallP) row = min(row, P - 1);
      kr[e] = *reinterpret_cast<const u32x2*>(kb + (size_t)(ws + row) * D + dq * 4);
    }
    wait_vmcnt<0>();
    // K^T: tokens outside [lo, hi) contribute zero
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = dq * 4 + c;
      uint32_t w[KPT / 2];
#pragma unroll
      for (int e = 0; e < KPT / 2; ++e) {
        const int r0 = kg * KPT + 2 * e;
        const uint32_t x0 = c < 2 ? kr[2 * e].x : kr[2 * e].y;
        const uint32_t x1 = c < 2 ? kr[2 * e + 1].x : kr[2 * e + 1].y;
        const uint32_t h0 = (c & 1) ? (x0 >> 16) : (x0 & 0xffffu);
        const uint32_t h1 = (c & 1) ? (x1 >> 16) : (x1 & 0xffffu);
        const bool ok0 = r0 >= lo && r0 < hi, ok1 = r0 + 1 >= lo && r0 + 1 < hi;
        w[e] = (ok0 ? h0 : 0u) | ((ok1 ? h1 : 0u) << 16);
      }
      const int key0 = kg * KPT;
      uint8_t* dst = &sm.kt[d * kRow + (((key0 >> 3) ^ swz(d)) << 4) + (key0 & 7) * 2];
      if constexpr (KPT == 8) *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
      else *reinterpret_cast<u32x2*>(dst) = u32x2{w[0], w[1]};
    }
    __syncthreads();
    if (lo > 0 || hi < kT) {
      // E_V^T: the same tokens contribute zero to cv
      for (int x = tid; x < R * kT; x += 256) {
        const int j = x / kT, t = x % kT;
        if (t < lo || t >= hi)
          *reinterpret_cast<uint16_t*>(&sm.ev[j * kRow + (((t >> 3) ^ swz(j)) << 4) + (t & 7) * 2]) = 0;
      }
      __syncthreads();
    }
#pragma unroll
    for (int ks = 0; ks < kT / 16; ++ks) {
      const int chunk = 2 * ks + (lane >> 5);
#pragma unroll
      for (int q = 0; q < TPW; ++q) {
        const int ti = wave * TPW + q;
        const uint8_t *ta, *tb;
        int ra, rb;
        if (ti < NTK) {  // ck[j][d] += E_K^T[j][t] K^T[d][t]
          ra = (ti / NMD) * 32 + (lane & 31);
          rb = (ti % NMD) * 32 + (lane & 31);
          ta = sm.ek;
          tb = sm.kt;
        } else {         // cv[d][j] += V[d][t] E_V^T[j][t]
          ra = ((ti - NTK) / NMR) * 32 + (lane & 31);
          rb = ((ti - NTK) % NMR) * 32 + (lane & 31);
          ta = sm.vt;
          tb = sm.ev;
        }
        const u32x4 a = ld_lds16(ta + ra * kRow + ((chunk ^ swz(ra)) << 4));
        const u32x4 bb = ld_lds16(tb + rb * kRow + ((chunk ^ swz(rb)) << 4));
        acc[q] = mfma32(a, bb, acc[q]);
      }
    }
    __syncthreads();
  }

  // lane holds column (lane % 32) of each output tile, rows 8(r/4) + 4(lane/32) + r%4
  uint16_t* ck = static_cast<uint16_t*>(p.ck) + hb * R * D;   // [R][D]
  uint16_t* cv = static_cast<uint16_t*>(p.cv) + hb * D * R;   // [D][R]
  float* part_out = p.parts > 1
      ? p.partial + ((((size_t)b * p.H + h) * p.n_pages + pi) * p.parts + part) * (2 * R * D)
      : nullptr;
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    const int ti = wave * TPW + q;
    const bool is_k = ti < NTK;
    const int mt = is_k ? ti / NMD : (ti - NTK) / NMR;
    const int nt = is_k ? ti % NMD : (ti - NTK) % NMR;
    const int ncols = is_k ? D : R;
    const int col = nt * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = mt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const size_t e = (size_t)row * ncols + col;
      if (part_out) {
        part_out[(is_k ? 0 : R * D) + e] = acc[q][r];
      } else {
        const uint16_t v = (uint16_t)(pack_bf16(acc[q][r], 0.f) & 0xffffu);
        if (is_k) ck[e] = v;
        else cv[e] = v;
      }
    }
  }
}

// Sum of a page's parts in part order, rounded once to bf16. One workgroup
// per (1024 outputs, page, head), four consecutive outputs per thread.
constexpr int kReduceChunk = 1024;

__global__ __launch_bounds__(256) void compress_reduce_kernel(CompressParams p) {
  const int RD = p.R * p.D;
  const int chunks = 2 * RD / kReduceChunk;
  const int pi = blockIdx.x / chunks, c = blockIdx.x % chunks, h = blockIdx.y, b = blockIdx.z;
  const int page = p.first_page + pi;
  const int slot = clampi(p.page_table[(size_t)b * p.max_pages + page], 0, p.num_slots - 1);
  const size_t hb = (size_t)slot * p.H + h;
  const float* src = p.partial + (((size_t)b * p.H + h) * p.n_pages + pi) * p.parts * (2 * RD);
  const int e = c * kReduceChunk + 4 * threadIdx.x;
  f32x4 s = *reinterpret_cast<const f32x4*>(src + e);
  for (int k = 1; k < p.parts; ++k) s += *reinterpret_cast<const f32x4*>(src + (size_t)k * 2 * RD + e);
  uint16_t* dst = (e < RD ? static_cast<uint16_t*>(p.ck) + hb * RD + e
                          : static_cast<uint16_t*>(p.cv) + hb * RD + (e - RD));
  *reinterpret_cast<u32x2*>(dst) = u32x2{pack_bf16(s.x, s.y), pack_bf16(s.z, s.w)};
}

// fp32 inputs: plain VALU products, fp32 accumulation in token order (small
// shapes; fp32 end to end).
__global__ __launch_bounds__(256) void compress_f32_kernel(CompressParams p) {
  const int pi = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int page = p.first_page + pi;
  const int slot = clampi(p.page_table[(size_t)b * p.max_pages + page], 0, p.num_slots - 1);
  const size_t hb = (size_t)slot * p.H + h;
  const int P = p.P, R = p.R, D = p.D;
  const float* kb = static_cast<const float*>(p.k) + hb * P * D;
  const float* vb = static_cast<const float*>(p.v) + hb * D * P;
  const float* ekb = static_cast<const float*>(p.e_k) + (size_t)h * R * P;
  const float* evb = static_cast<const float*>(p.e_v) + (size_t)h * R * P;
  float* ck = static_cast<float*>(p.ck) + hb * R * D;
  float* cv = static_cast<float*>(p.cv) + hb * D * R;
  for (int e = threadIdx.x; e < 2 * R * D; e += 256) {
    float s = 0.f;
    if (e < R * D) {
      const int j = e / D, d = e % D;
      for (int t = 0; t < P; ++t) s = fmaf(ekb[(size_t)j * P + t], kb[(size_t)t * D + d], s);
      ck[e] = s;
    } else {
      const int d = (e - R * D) / R, j = (e - R * D) % R;
      for (int t = 0; t < P; ++t) s = fmaf(vb[(size_t)d * P + t], evb[(size_t)j * P + t], s);
      cv[e - R * D] = s;
    }
  }
}

template <int D, int R>
void launch_compress_bf16(const CompressParams& p, int B, hipStream_t s) {
  const dim3 grid(p.n_pages * p.parts, p.H, B);
  if (p.P < kT) compress_bf16_kernel<D, R, true><<<grid, 256, 0, s>>>(p);
  else compress_bf16_kernel<D, R, false><<<grid, 256, 0, s>>>(p);
}

}  // namespace

hipError_t launch_compress(int dtype, int B, const CompressParams& p, hipStream_t s) {
  if (dtype != HSA_DTYPE_BF16) {
    compress_f32_kernel<<<dim3(p.n_pages, p.H, B), 256, 0, s>>>(p);
    return hipGetLastError();
  }
  if (p.D == 128) {
    if (p.R == 32) launch_compress_bf16<128, 32>(p, B, s);
    else if (p.R == 64) launch_compress_bf16<128, 64>(p, B, s);
    else launch_compress_bf16<128, 128>(p, B, s);
  } else {
    if (p.R == 32) launch_compress_bf16<64, 32>(p, B, s);
    else if (p.R == 64) launch_compress_bf16<64, 64>(p, B, s);
    else launch_compress_bf16<64, 128>(p, B, s);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.parts == 1) return e;
  // 2 R d is a multiple of kReduceChunk for every supported (R, d)
  compress_reduce_kernel<<<dim3(p.n_pages * (2 * p.R * p.D / kReduceChunk), p.H, B), 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace hsa

// Linear-branch state and page index: one streaming pass over the new pages.
//
// For the pages being folded in, every (batch, head) accumulates
//   kv_state[j][i] += sum_t phi(k_t)[i] v_t[j],  k_state[i] += sum_t phi(k_t)[i]
// (kernelised linear branch, feature map elu+1) and the mean key of each page
// (Sec. 3.2, Stage-2 page index) in fp64.
//
// The pass is HBM-bound (512 bytes read per key and head against 2*d*d
// flops, well below the MFMA ridge), so the kernel is built around keeping
// loads in flight: value pages (stored d-major) go straight from HBM into LDS
// with global_load_lds, key rows come through registers because they must be
// transposed (the contraction runs over keys, so both MFMA operands need
// keys contiguous) and mapped through phi on the way. The contraction is
// bf16 MFMA with fp32 accumulation; partial states per workgroup are reduced
// in a fixed order by a second kernel (deterministic, no atomics).
#include <type_traits>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

constexpr int kTileKeys = 64;          // keys per LDS tile
constexpr int kRowBytes = kTileKeys * 2;  // one LDS row: 64 bf16 keys

// LDS rows of 8 x 16-byte chunks; XOR swizzle so that 16 consecutive rows
// read at the same logical chunk hit distinct bank groups.
__device__ __forceinline__ int swz8(int row) { return ((row >> 1) ^ (row >> 4)) & 7; }

constexpr int kUnitsPerBatch = 8;       // page sums staged in LDS per batch

template <int D>
struct StateSmem {
  uint8_t vt[3][D * kRowBytes];   // V^T tiles: [d_v][64 keys] bf16, 3-stage ring
  uint8_t fk[D * kRowBytes];      // phi(K)^T tile: [d_k][64 keys] bf16
  double red[8 * 128];            // cross-thread reductions (8 KB)
  double ksum[kUnitsPerBatch * D];  // key sums of the batch's units
};

// One workgroup folds units [u_begin, u_end) of one (batch, head); a unit is
// one part of one page. Units go in batches of up to kUnitsPerBatch; the
// 64-key tiles of a batch run as one flat sequence across unit boundaries.
// While tile t is converted and contracted, K rows of tile t+1 (registers)
// and V^T tiles t+1 and t+2 (3-slot LDS ring) are in flight. No global
// store and no branch around a load happens inside that loop, and the
// single register set keeps the load order fixed, so the only vector-memory
// wait there is the in-order one that leaves the newest V tile in flight;
// the batch's page sums are kept in LDS and written once it is done.
template <int D, bool kSmallP>
__global__ __launch_bounds__(256, 2) void state_bf16_kernel(StateParams p) {
  constexpr int DQ = D / 4;                // 4-wide d groups per key row
  constexpr int KG = 256 / DQ;             // key groups
  constexpr int KPT = kTileKeys / KG;      // keys per thread per tile (8 or 4)
  constexpr int NV = D / 32;               // V^T 1-KB load instructions per wave
  constexpr int NT = D / 32;               // 32-wide output blocks per dim
  constexpr int TPW = NT * NT / 4;         // output tiles per wave
  static_assert(KPT == 8 || KPT == 4, "layout");
  __shared__ __attribute__((aligned(16))) StateSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = blockIdx.x / p.n_groups, grp = blockIdx.x % p.n_groups;
  const int b = bh / p.H, h = bh % p.H;
  const int n_units = p.n_pages * p.parts;
  const int u_begin = grp * p.upw;
  const int u_end = min(n_units, u_begin + p.upw);  // the plan gives every group >= 1 unit

  const uint16_t* __restrict__ kb = static_cast<const uint16_t*>(p.k);
  const uint16_t* __restrict__ vb = static_cast<const uint16_t*>(p.v);
  const int dq = tid % DQ, kg = tid / DQ;  // K-load role: 4 dims x KPT keys
  const int tiles_full = (p.part_len + kTileKeys - 1) / kTileKeys;

  // key range of unit u
  auto unit_keys = [&](int u, int& k_beg, int& k_end) {
    k_beg = (u % p.parts) * p.part_len;
    k_end = min(p.P, k_beg + p.part_len);
  };
  auto unit_tiles = [&](int u) {
    int k_beg, k_end;
    unit_keys(u, k_beg, k_end);
    return k_end - k_beg < p.part_len ? (k_end - k_beg + kTileKeys - 1) / kTileKeys : tiles_full;
  };
  auto head_base = [&](int u) {
    const int page = p.first_page + u / p.parts;
    const int slot = clampi(ld_const(p.page_table + (size_t)b * p.max_pages + page), 0, p.num_slots - 1);
    return (size_t)slot * p.H + h;
  };

  // Per-lane byte offsets of the tile loads, fixed for the whole pass: V^T
  // rows (8 keys at swizzled chunk c of d-row r, relative to the tile's
  // first key) and K rows (KPT keys x 4 dims). A tile then costs one scalar
  // base per tensor.
  uint32_t v_off[NV], k_off[KPT];
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    const int r = (wave * NV + n) * 8 + (lane >> 3);
    v_off[n] = (uint32_t)(r * p.P + 8 * ((lane & 7) ^ swz8(r))) * 2u;
  }
#pragma unroll
  for (int e = 0; e < KPT; ++e) k_off[e] = (uint32_t)((kg * KPT + e) * D + dq * 4) * 2u;

  f32x16 acc[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) acc[t] = f32x16{0};
  float zacc[4] = {0.f, 0.f, 0.f, 0.f};

  for (int ub = u_begin; ub < u_end; ub += kUnitsPerBatch) {
    const int ue = min(u_end, ub + kUnitsPerBatch);
    int total = 0;
    for (int u = ub; u < ue; ++u) total += unit_tiles(u);

    // Two cursors: K rows run one tile ahead (one register set), V^T tiles
    // two tiles ahead (3-slot LDS ring). Each step issues K(t+1) first, then
    // V(t+2), so waiting for K(t+1) at the next step leaves V(t+2) in flight.
    struct Cursor { int u, t, n; };
    auto cur_init = [&](Cursor& c) { c.u = ub; c.t = 0; c.n = unit_tiles(ub); };
    auto cur_next = [&](Cursor& c) {   // stays on the batch's last tile
      if (c.t + 1 < c.n) ++c.t;
      else if (c.u + 1 < ue) { ++c.u; c.t = 0; c.n = unit_tiles(c.u); }
    };
    // Source window of a tile: 64 keys ending at the unit's end when fewer
    // remain (every unit ends at key >= 64 when P >= 64), so that its loads
    // are one scalar base plus the constant per-lane offsets; rows before
    // the tile's first key are masked when converted. Pages shorter than a
    // tile (kSmallP) clamp per lane instead.
    auto tile_src = [&](const Cursor& c, int& ws, int& nv, size_t& hb) {
      int k_beg, k_end;
      unit_keys(c.u, k_beg, k_end);
      const int k0 = k_beg + c.t * kTileKeys;
      nv = min(kTileKeys, k_end - k0);
      ws = kSmallP ? k0 : min(k0, k_end - kTileKeys);
      hb = head_base(c.u);
    };
    auto issue_k = [&](u32x2 (&kr)[KPT], const Cursor& c) {
      int ws, nv; size_t hb;
      tile_src(c, ws, nv, hb);
      const char* ksrc = reinterpret_cast<const char*>(kb + (hb * p.P + ws) * D); // [P][D]
#pragma unroll
      for (int e = 0; e < KPT; ++e) {
        uint32_t off = k_off[e];
        if constexpr (kSmallP) off -= (uint32_t)(max(0, kg * KPT + e - (nv - 1)) * D * 2);
        kr[e] = *reinterpret_cast<const u32x2*>(ksrc + off);
      }
    };
    auto issue_v = [&](const Cursor& c, int slot_v) {
      int ws, nv; size_t hb;
      tile_src(c, ws, nv, hb);
      const char* vsrc = reinterpret_cast<const char*>(vb + hb * D * p.P + ws);   // [D][P]
      uint8_t* vdst = &sm.vt[slot_v][wave * NV * 1024];
#pragma unroll
      for (int n = 0; n < NV; ++n) {
        uint32_t off = v_off[n];
        if constexpr (kSmallP) {
          const int r = (wave * NV + n) * 8 + (lane >> 3);
          off -= (uint32_t)(max(0, 8 * ((lane & 7) ^ swz8(r)) - (nv - 8)) * 2);
        }
        g2lds16(vsrc + off, vdst + n * 1024);
      }
    };

    Cursor ck, cv;
    cur_init(ck);
    cur_init(cv);
    u32x2 kr[KPT];
    issue_v(cv, 0); cur_next(cv);
    issue_k(kr, ck); cur_next(ck);
    issue_v(cv, 1); cur_next(cv);

    // consume cursor
    int cu = ub, ct = 0, cu_tiles = unit_tiles(ub);
    double kacc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int t = 0; t < total; ++t) {
      wait_vmcnt<NV>();                   // K(t) and V(t) have landed; V(t+1) may be in flight
      __builtin_amdgcn_sched_barrier(0);
      // valid rows of this tile's window: [lo, hi)
      int k_beg, k_end;
      unit_keys(cu, k_beg, k_end);
      const int k0 = k_beg + ct * kTileKeys;
      const int nv = min(kTileKeys, k_end - k0);
      const int lo = kSmallP ? 0 : k0 - min(k0, k_end - kTileKeys);
      const int hi = kSmallP ? nv : kTileKeys;
      float f[KPT][4];
      auto convert = [&](auto full) {
#pragma unroll
        for (int e = 0; e < KPT; ++e) {
          const int row = kg * KPT + e;
          const bool ok = decltype(full)::value || (row >= lo && row < hi);
          const float x[4] = {bf16_lo(kr[e].x), bf16_hi(kr[e].x), bf16_lo(kr[e].y), bf16_hi(kr[e].y)};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const float y = ok ? phi(x[c]) : 0.f;
            f[e][c] = y;
            zacc[c] += y;
            kacc[c] += ok ? (double)x[c] : 0.0;
          }
        }
      };
      if (nv == kTileKeys) convert(std::true_type{});
      else convert(std::false_type{});
      lds_barrier();
      issue_k(kr, ck); cur_next(ck);
      issue_v(cv, (t + 2) % 3); cur_next(cv);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int row = dq * 4 + c;
        uint32_t w[KPT / 2];
#pragma unroll
        for (int e = 0; e < KPT / 2; ++e) w[e] = pack_bf16(f[2 * e][c], f[2 * e + 1][c]);
        const int key0 = kg * KPT;
        const int chunk = key0 >> 3, within = (key0 & 7) * 2;
        uint8_t* dst = &sm.fk[row * kRowBytes + ((chunk ^ swz8(row)) << 4) + within];
        if constexpr (KPT == 8) {
          *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
        } else {
          *reinterpret_cast<u32x2*>(dst) = u32x2{w[0], w[1]};
        }
      }
      lds_barrier();
      const uint8_t* vt = sm.vt[t % 3];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int chunk = 2 * ks + (lane >> 5);
#pragma unroll
        for (int q = 0; q < TPW; ++q) {
          const int ti = wave * TPW + q;
          const int mj = ti / NT, ni = ti % NT;
          const int ra = mj * 32 + (lane & 31);
          const int rb = ni * 32 + (lane & 31);
          const u32x4 a = ld_lds16(vt + ra * kRowBytes + ((chunk ^ swz8(ra)) << 4));
          const u32x4 bb = ld_lds16(sm.fk + rb * kRowBytes + ((chunk ^ swz8(rb)) << 4));
          acc[q] = mfma32(a, bb, acc[q]);
        }
      }
      if (++ct == cu_tiles) {
#pragma unroll
        for (int c = 0; c < 4; ++c) sm.red[kg * D + dq * 4 + c] = kacc[c];
        lds_barrier();
        if (tid < D) {
          double s = 0.0;
          for (int g = 0; g < KG; ++g) s += sm.red[g * D + tid];
          sm.ksum[(cu - ub) * D + tid] = s;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) kacc[c] = 0.0;
        ++cu;
        ct = 0;
        if (cu < ue) cu_tiles = unit_tiles(cu);
      }
    }
    // the trailing re-reads (the cursors stay on the batch's last tile)
    // complete before the ring is reused or the workgroup's LDS is released;
    // then the batch's page sums go out
    wait_vmcnt<0>();
    __syncthreads();
    double* dst = p.ws_k + ((size_t)bh * n_units + ub) * D;
    for (int x = tid; x < (ue - ub) * D; x += 256) dst[x] = sm.ksum[x];
    wait_vmcnt<0>();
    __syncthreads();
  }

  // normaliser partial
  float* redf = reinterpret_cast<float*>(sm.red);
#pragma unroll
  for (int c = 0; c < 4; ++c) redf[kg * D + dq * 4 + c] = zacc[c];
  __syncthreads();
  const size_t g_index = (size_t)bh * p.n_groups + grp;
  if (tid < D) {
    float s = 0.f;
    for (int g = 0; g < KG; ++g) s += redf[g * D + tid];
    p.ws_z[g_index * D + tid] = s;
  }
  // state partial: lane holds column i = 32 ni + lane%32, rows j of the tile
  float* out = p.ws_S + g_index * D * D;
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    const int ti = wave * TPW + q;
    const int mj = ti / NT, ni = ti % NT;
    const int i = ni * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = mj * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      out[j * D + i] = acc[q][r];
    }
  }
}

// fp32 inputs: plain VALU contraction (small shapes; fp32 end to end).
template <int D>
__global__ __launch_bounds__(256) void state_f32_kernel(StateParams p) {
  constexpr int T = 32;
  constexpr int EPT = D * D / 256;  // state elements per thread (contiguous i)
  __shared__ float fk[T][D + 1];
  __shared__ float vt[D][T + 1];
  __shared__ float kraw[T][D + 1];
  const int tid = threadIdx.x;
  const int bh = blockIdx.x / p.n_groups, grp = blockIdx.x % p.n_groups;
  const int b = bh / p.H, h = bh % p.H;
  const int n_units = p.n_pages * p.parts;
  const int u_begin = grp * p.upw, u_end = min(n_units, u_begin + p.upw);
  const float* kb = static_cast<const float*>(p.k);
  const float* vb = static_cast<const float*>(p.v);
  const int j = (tid * EPT) / D, i0 = (tid * EPT) % D;
  float acc[EPT];
  for (int e = 0; e < EPT; ++e) acc[e] = 0.f;
  float zacc = 0.f;
  for (int u = u_begin; u < u_end; ++u) {
    const int page = p.first_page + u / p.parts, part = u % p.parts;
    const int k_beg = part * p.part_len, k_end = min(p.P, k_beg + p.part_len);
    const int slot = clampi(p.page_table[(size_t)b * p.max_pages + page], 0, p.num_slots - 1);
    const size_t head_base = (size_t)slot * p.H + h;
    const float* kpage = kb + head_base * p.P * D;
    const float* vpage = vb + head_base * D * p.P;
    double kacc = 0.0;
    for (int k0 = k_beg; k0 < k_end; k0 += T) {
      const int nk = min(T, k_end - k0);
      __syncthreads();
      for (int x = tid; x < T * D; x += 256) {
        const int key = x / D, dd = x % D;
        const float kv = key < nk ? kpage[(size_t)(k0 + key) * D + dd] : 0.f;
        kraw[key][dd] = kv;
        fk[key][dd] = key < nk ? phi(kv) : 0.f;
      }
      for (int x = tid; x < T * D; x += 256) {
        const int dd = x / T, key = x % T;
        vt[dd][key] = key < nk ? vpage[(size_t)dd * p.P + k0 + key] : 0.f;
      }
      __syncthreads();
      if (tid < D) {
        for (int key = 0; key < nk; ++key) {
          kacc += (double)kraw[key][tid];
          zacc += fk[key][tid];
        }
      }
      for (int key = 0; key < nk; ++key) {
        const float vv = vt[j][key];
        for (int e = 0; e < EPT; ++e) acc[e] += vv * fk[key][i0 + e];
      }
    }
    if (tid < D) p.ws_k[((size_t)bh * n_units + u) * D + tid] = kacc;
  }
  const size_t g_index = (size_t)bh * p.n_groups + grp;
  if (tid < D) p.ws_z[g_index * D + tid] = zacc;
  for (int e = 0; e < EPT; ++e) p.ws_S[g_index * D * D + j * D + i0 + e] = acc[e];
}

// Fixed-order reduction of the partials into the caller's state: each thread
// owns 16 bytes of the output and adds the partials in increasing order,
// eight loads in flight at a time.
typedef double f64x2 __attribute__((ext_vector_type(2)));

template <typename V>
__device__ __forceinline__ V sum_groups(const V* src, size_t stride, int n) {
  V s = V{0};
  int g = 0;
  for (; g + 8 <= n; g += 8) {
    V x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = src[(size_t)(g + u) * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += x[u];
  }
  for (; g < n; ++g) s += src[(size_t)g * stride];
  return s;
}

template <int D>
__global__ __launch_bounds__(256) void state_reduce_kernel(StateReduceParams r) {
  constexpr int nS = D * D / 4, nz = D / 4;  // in float4 units
  const int bh = blockIdx.x;
  const int e = blockIdx.y * 256 + threadIdx.x;
  const int nk = r.n_pages * D / 2;          // in double2 units
  if (e < nS) {
    const f32x4* src = reinterpret_cast<const f32x4*>(r.ws_S) + (size_t)bh * r.n_groups * nS + e;
    f32x4* dst = reinterpret_cast<f32x4*>(r.kv_state) + (size_t)bh * nS + e;
    *dst += sum_groups(src, nS, r.n_groups);
  } else if (e < nS + nz) {
    const int i = e - nS;
    const f32x4* src = reinterpret_cast<const f32x4*>(r.ws_z) + (size_t)bh * r.n_groups * nz + i;
    f32x4* dst = reinterpret_cast<f32x4*>(r.k_state) + (size_t)bh * nz + i;
    *dst += sum_groups(src, nz, r.n_groups);
  } else if (e < nS + nz + nk) {
    const int x = e - nS - nz;
    const int pg = x / (D / 2), dd = x % (D / 2);
    const f64x2* src = reinterpret_cast<const f64x2*>(r.ws_k) + ((size_t)bh * r.n_pages + pg) * r.parts * (D / 2) + dd;
    const f64x2 s = sum_groups(src, D / 2, r.parts);
    f64x2* dst = reinterpret_cast<f64x2*>(r.page_kmean) + ((size_t)bh * r.max_pages + r.first_page + pg) * (D / 2) + dd;
    *dst = s / (double)r.P;
  }
}

}  // namespace

hipError_t launch_state_update(int dtype, int d, int B, const StateParams& p,
                               const StateReduceParams& r, hipStream_t s) {
  const dim3 grid(B * p.H * p.n_groups);
  if (dtype == HSA_DTYPE_BF16) {
    const bool small = p.P < kTileKeys;
    if (d == 128) {
      if (small) state_bf16_kernel<128, true><<<grid, 256, 0, s>>>(p);
      else state_bf16_kernel<128, false><<<grid, 256, 0, s>>>(p);
    } else {
      if (small) state_bf16_kernel<64, true><<<grid, 256, 0, s>>>(p);
      else state_bf16_kernel<64, false><<<grid, 256, 0, s>>>(p);
    }
  } else {
    if (d == 128) state_f32_kernel<128><<<grid, 256, 0, s>>>(p);
    else state_f32_kernel<64><<<grid, 256, 0, s>>>(p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int total = d * d / 4 + d / 4 + p.n_pages * d / 2;
  const dim3 rgrid(B * p.H, (total + 255) / 256);
  if (d == 128) state_reduce_kernel<128><<<rgrid, 256, 0, s>>>(r);
  else state_reduce_kernel<64><<<rgrid, 256, 0, s>>>(r);
  return hipGetLastError();
}

}  // namespace hsa

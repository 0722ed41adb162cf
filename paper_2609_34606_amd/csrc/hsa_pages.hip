// Page append: new keys and values of a chunk, token-major as a projection
// writes them, copied into their pool slots in the pool's layouts (key pages
// [P][d], value pages d-major [d][P]), optionally in cube order.
//
// Cube order (App. "Block Sparse Attention", the flattening index of
// (C_t, C_h, C_w) cubes): the tokens of a page of T frames x H x W are
// stored cube by cube, so that a run of B = C_t C_h C_w consecutive stored
// tokens is one spatio-temporal cube, and a key block of the head-adaptive
// sparse branch is a cube. The paper assumes that the cube divides the
// latent; at 480p a frame is 30 x 52 tokens, so H = 30 is not a multiple of
// C_h = 8 (or 4). Cubes that fit whole come first, in the paper's order
// (cube t index, then h, then w; tokens in (t, h, w) order inside a cube);
// the truncated cubes along the far edges follow in the same order. When the
// extents divide, this is exactly the paper's index.
#include <algorithm>

#include "hsa_device.h"
#include "hsa_kernels.h"

namespace hsa {
namespace {

constexpr int kTok = 64;  // tokens per workgroup

// One (b, new page, head, 64-token run) per workgroup: keys row by row,
// values through LDS to the d-major page layout.
template <typename T, int D>
__global__ __launch_bounds__(256) void page_write_kernel(PageWriteParams p) {
  __shared__ T vs[kTok][D + (sizeof(T) == 2 ? 2 : 1)];
  const int tid = threadIdx.x;
  const int run = blockIdx.x, h = blockIdx.y;
  const int b = blockIdx.z / p.n_pages, pg = blockIdx.z % p.n_pages;
  const int i0 = run * kTok;
  const int n = min(kTok, p.P - i0);
  const int slot = clampi(ld_const(p.page_table + (size_t)b * p.max_pages + p.first_page + pg), 0,
                          p.num_slots - 1);
  const T* ksrc = static_cast<const T*>(p.k_src);
  const T* vsrc = static_cast<const T*>(p.v_src);
  T* kdst = static_cast<T*>(p.k) + ((size_t)slot * p.H + h) * p.P * D;
  T* vdst = static_cast<T*>(p.v) + ((size_t)slot * p.H + h) * D * p.P;
  // source row of stored token i: token src_of[i] of the page in raster order
  auto src_row = [&](int i) {
    const int s = p.src_of ? clampi(p.src_of[i], 0, p.P - 1) : i;
    return (((size_t)b * p.n_pages + pg) * p.P + s) * p.H + h;
  };
  for (int e = tid; e < n * D; e += 256) {
    const int i = e / D, c = e % D;
    const size_t r = src_row(i0 + i);
    kdst[(size_t)(i0 + i) * D + c] = ksrc[r * D + c];
    vs[i][c] = vsrc[r * D + c];
  }
  __syncthreads();
  for (int e = tid; e < n * D; e += 256) {
    const int c = e / n, i = e % n;
    vdst[(size_t)c * p.P + i0 + i] = vs[i][c];
  }
}

}  // namespace

hipError_t launch_page_write(int dtype, int d, int B, const PageWriteParams& p, hipStream_t s) {
  const dim3 grid((p.P + kTok - 1) / kTok, p.H, B * p.n_pages);
  if (dtype == HSA_DTYPE_BF16) {
    if (d == 128) page_write_kernel<uint16_t, 128><<<grid, 256, 0, s>>>(p);
    else page_write_kernel<uint16_t, 64><<<grid, 256, 0, s>>>(p);
  } else {
    if (d == 128) page_write_kernel<float, 128><<<grid, 256, 0, s>>>(p);
    else page_write_kernel<float, 64><<<grid, 256, 0, s>>>(p);
  }
  return hipGetLastError();
}

int cube_order(int T, int H, int W, int ct, int ch, int cw, int32_t* src_of) {
  const int Nt = T / ct, Nh = H / ch, Nw = W / cw;                    // whole cubes
  const int Mt = (T + ct - 1) / ct, Mh = (H + ch - 1) / ch, Mw = (W + cw - 1) / cw;
  int n = 0;
  auto emit_cube = [&](int a, int bh, int c) {
    for (int t = a * ct; t < std::min(T, (a + 1) * ct); ++t)
      for (int hh = bh * ch; hh < std::min(H, (bh + 1) * ch); ++hh)
        for (int w = c * cw; w < std::min(W, (c + 1) * cw); ++w) src_of[n++] = (t * H + hh) * W + w;
  };
  for (int a = 0; a < Nt; ++a)
    for (int bh = 0; bh < Nh; ++bh)
      for (int c = 0; c < Nw; ++c) emit_cube(a, bh, c);
  const int whole = n;
  for (int a = 0; a < Mt; ++a)
    for (int bh = 0; bh < Mh; ++bh)
      for (int c = 0; c < Mw; ++c)
        if (a >= Nt || bh >= Nh || c >= Nw) emit_cube(a, bh, c);
  return whole;
}

}  // namespace hsa

// Host tier of the context store (paper section 3.2.2, "Layered Storage of
// Action Context": rarely used context moves to CPU memory): copies of whole
// rows between the K/V page pools and pinned host memory, written and read by
// the kernels themselves through the host buffers' device addresses.
//
// Host image of a row (after a 256-byte header the host fills):
//   K/V  [layer][K|V][head][len][head_dim]   compute type
//   h_last [d] fp32, then its fp16 pair hi [d], lo [d]
// One workgroup per (row, layer, K|V, head) moves that head's len x head_dim
// values (contiguous on the host side, 64-position runs on the device side);
// one more per row moves the hidden state of its last position.
#include "common.h"
#include "kernels.h"

namespace ams {

namespace {

template <bool TO_HOST>
__global__ __launch_bounds__(256) void k_rows_xfer(const XferRow* __restrict__ rows, int n_rows, int L, int H,
                                                   int dh, int es, char* __restrict__ pool, size_t slab_layer,
                                                   const int32_t* __restrict__ pt, int ppr, float* __restrict__ h_last,
                                                   f16* __restrict__ h16, f16* __restrict__ h16lo, int d) {
  const int per_row = 2 * L * H + 1;
  const int i = blockIdx.x / per_row, k = blockIdx.x % per_row;
  if (i >= n_rows) return;
  const XferRow xr = rows[i];
  char* host = (char*)xr.host + 256;
  const size_t head_bytes = (size_t)xr.len * dh * es;  // one (layer, K|V, head) on the host
  if (k == 2 * L * H) {  // the last position's hidden state (+ its fp16 pair)
    float* hh = (float*)(host + (size_t)2 * L * H * head_bytes);
    f16* hp = (f16*)(hh + d);
    for (int e = threadIdx.x; e < d; e += blockDim.x) {
      const size_t o = (size_t)xr.row * d + e;
      if (TO_HOST) {
        hh[e] = h_last[o];
        hp[e] = h16[o];
        hp[d + e] = h16lo[o];
      } else {
        h_last[o] = hh[e];
        h16[o] = hp[e];
        h16lo[o] = hp[d + e];
      }
    }
    return;
  }
  const int l = k / (2 * H), kv = (k / H) % 2, h = k % H;
  char* layer = pool + (size_t)(2 * l + kv) * slab_layer;
  char* hp = host + (size_t)((l * 2 + kv) * H + h) * head_bytes;
  const int cpp = dh * es / 16;  // 16-byte chunks per position
  const int32_t* prow = pt + (size_t)xr.row * ppr;
  for (int q = threadIdx.x; q < xr.len * cpp; q += blockDim.x) {
    const int pos = q / cpp, c = q % cpp;
    const size_t dev = ((((size_t)prow[pos >> 6] * H + h) * KV_PAGE + (pos & (KV_PAGE - 1))) * dh) * es + 16 * c;
    uint4* dp = (uint4*)(layer + dev);
    uint4* hq = (uint4*)(hp + (size_t)q * 16);
    if (TO_HOST) *hq = *dp;
    else *dp = *hq;
  }
}

}  // namespace

hipError_t rows_xfer(bool to_host, const XferRow* rows, int n_rows, int L, int H, int dh, int es, void* pool,
                     size_t slab_layer, const int32_t* pt, int ppr, float* h_last, void* h16, void* h16lo, int d,
                     hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)(n_rows * (2 * L * H + 1)));
  if (to_host)
    hipLaunchKernelGGL(k_rows_xfer<true>, grid, dim3(256), 0, s, rows, n_rows, L, H, dh, es, (char*)pool, slab_layer,
                       pt, ppr, h_last, (f16*)h16, (f16*)h16lo, d);
  else
    hipLaunchKernelGGL(k_rows_xfer<false>, grid, dim3(256), 0, s, rows, n_rows, L, H, dh, es, (char*)pool,
                       slab_layer, pt, ppr, h_last, (f16*)h16, (f16*)h16lo, d);
  return hipGetLastError();
}

}  // namespace ams

// Row-wise kernels: RMSNorm, embedding gathers, prefix ingest, weight
// packing, the RoPE table, last-token gathers and length bookkeeping.
#include "common.h"
#include "kernels.h"

namespace ams {

// One workgroup per token row (256 threads up to d = 4096, else 1024);
// statistics in fp32.  Each thread loads its EPT (<= 16) elements before
// reducing, so a row costs one memory round trip.
template <typename T, int EPT>
__global__ __launch_bounds__(1024) void k_rmsnorm(const float* __restrict__ h, int d, float eps, T* __restrict__ u,
                                                  T* __restrict__ ulo) {
  __shared__ float red[16];
  const size_t base = (size_t)blockIdx.x * d;
  const int nt = blockDim.x;
  float x[EPT];
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = threadIdx.x + e * nt;
    x[e] = i < d ? h[base + i] : 0.f;
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) ss = fmaf(x[e], x[e], ss);
  const float tot = block_sum(ss, red);
  const float rs = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = threadIdx.x + e * nt;
    if (i < d) {
      if constexpr (sizeof(T) == 2) split16(x[e] * rs, u, ulo, base + i);
      else st<T>(u, base + i, x[e] * rs);
    }
  }
}

template <typename T>
static hipError_t rmsnorm_t(const float* h, int M, int d, float eps, T* u, T* ulo, hipStream_t s) {
  const int nt = d <= 4096 ? 256 : 1024;
  const int ept = (d + nt - 1) / nt;  // <= 16 for d <= 16384
#define AMS_RMS(E) hipLaunchKernelGGL((k_rmsnorm<T, E>), dim3(M), dim3(nt), 0, s, h, d, eps, u, ulo)
  if (ept <= 1) AMS_RMS(1);
  else if (ept <= 2) AMS_RMS(2);
  else if (ept <= 4) AMS_RMS(4);
  else if (ept <= 8) AMS_RMS(8);
  else AMS_RMS(16);
#undef AMS_RMS
  return hipGetLastError();
}

hipError_t rmsnorm(int ct, const float* h, int M, int d, float eps, void* u, hipStream_t s, void* ulo) {
  if (M <= 0) return hipSuccess;
  if (ct == DT_F32) {
    if (ulo) return hipErrorInvalidValue;
    return rmsnorm_t<float>(h, M, d, eps, (float*)u, nullptr, s);
  }
  return rmsnorm_t<f16>(h, M, d, eps, (f16*)u, (f16*)ulo, s);
}

// h[m] += sum_s part[s][m] (splits added in order), then u[m] = fp16 of the
// new row over its rms: the split-K reduction of a token pass's residual
// projection with the next RMSNorm in the same pass over the row.  The norm
// sums the squares in k_rmsnorm's order, so u is bitwise what rmsnorm of the
// new h gives.
// S > 0: the split count as a constant, so every load of a thread (its h
// values and all their partial sums) is issued before the first add (with the
// count at run time the loads went out one element at a time: 40.8 us against
// 24 + 6.4 us for the two separate kernels at 1,024 x 4,096, 4 splits).
// S == 0 (counts the registers cannot hold at once): the splits go in groups
// of G, each group's loads for all the thread's elements issued together;
// a group's last loads past the split count read the last split again and are
// not added.
template <int EPT, int S>
__global__ __launch_bounds__(1024) void k_resid_norm(const float* __restrict__ part, int splits, int d, float eps,
                                                     float* __restrict__ h, f16* __restrict__ u) {
  __shared__ float red[16];
  const size_t base = (size_t)blockIdx.x * d, MN = (size_t)gridDim.x * d;
  const int nt = blockDim.x;
  constexpr int SP = S > 0 ? S : 1;
  float x[EPT], pv[EPT][SP];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = threadIdx.x + e * nt;
    x[e] = i < d ? h[base + i] : 0.f;
    if constexpr (S > 0) {
#pragma unroll
      for (int sp = 0; sp < S; ++sp) pv[e][sp] = i < d ? part[sp * MN + base + i] : 0.f;
    }
  }
  float acc[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) acc[e] = 0.f;
  if constexpr (S > 0) {
#pragma unroll
    for (int e = 0; e < EPT; ++e)
#pragma unroll
      for (int sp = 0; sp < S; ++sp) acc[e] += pv[e][sp];
  } else {
    constexpr int G = EPT >= 16 ? 2 : (EPT >= 8 ? 4 : 8);  // 32+ loads in flight, within 128 VGPRs
    for (int s0 = 0; s0 < splits; s0 += G) {
      float q[EPT][G];
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int i = threadIdx.x + e * nt, ic = i < d ? i : 0;
#pragma unroll
        for (int j = 0; j < G; ++j) q[e][j] = part[(size_t)min(s0 + j, splits - 1) * MN + base + ic];
      }
#pragma unroll
      for (int j = 0; j < G; ++j)
        if (s0 + j < splits)
#pragma unroll
          for (int e = 0; e < EPT; ++e) acc[e] += q[e][j];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = threadIdx.x + e * nt;
    if (i < d) {
      x[e] += acc[e];
      h[base + i] = x[e];
    }
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) ss = fmaf(x[e], x[e], ss);
  const float tot = block_sum(ss, red);
  const float rs = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = threadIdx.x + e * nt;
    if (i < d) u[base + i] = sat16(x[e] * rs);
  }
}

template <int EPT>
static void launch_resid_norm(const float* part, int splits, int M, int d, int nt, float* h, float eps, void* u,
                              hipStream_t s) {
#define AMS_RN(S_) \
  hipLaunchKernelGGL((k_resid_norm<EPT, S_>), dim3(M), dim3(nt), 0, s, part, splits, d, eps, h, (f16*)u)
  // (EPT * S partial sums in registers: at most 64, within the 128 VGPRs of 1,024 threads)
  switch (EPT * splits <= 64 ? splits : 0) {
    case 2: AMS_RN(2); break;
    case 3: AMS_RN(3); break;
    case 4: AMS_RN(4); break;
    case 8: if constexpr (EPT <= 8) { AMS_RN(8); break; } [[fallthrough]];
    default: AMS_RN(0); break;
  }
#undef AMS_RN
}

hipError_t resid_norm(const float* part, int splits, int M, int d, float* h, float eps, void* u, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (splits < 1) return hipErrorInvalidValue;
  const int nt = d <= 4096 ? 256 : 1024;  // as rmsnorm: the same sum of squares
  const int ept = (d + nt - 1) / nt;
  if (ept <= 1) launch_resid_norm<1>(part, splits, M, d, nt, h, eps, u, s);
  else if (ept <= 2) launch_resid_norm<2>(part, splits, M, d, nt, h, eps, u, s);
  else if (ept <= 4) launch_resid_norm<4>(part, splits, M, d, nt, h, eps, u, s);
  else if (ept <= 8) launch_resid_norm<8>(part, splits, M, d, nt, h, eps, u, s);
  else if (ept <= 16) launch_resid_norm<16>(part, splits, M, d, nt, h, eps, u, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Copies rows as raw elements (8/16-byte chunks); `ids` selects source rows.
template <typename T>
__global__ __launch_bounds__(256) void k_embed(const T* __restrict__ E, const int32_t* __restrict__ ids, int d,
                                               int vocab, T* __restrict__ out) {
  int id = ids[blockIdx.x];
  id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
  const T* src = E + (size_t)id * d;
  T* dst = out + (size_t)blockIdx.x * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = src[i];
}

hipError_t embed_rows(int st, const void* E, const int32_t* ids, int n, int d, int vocab, void* out,
                      hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (st == DT_F32)
    hipLaunchKernelGGL(k_embed<float>, dim3(n), dim3(256), 0, s, (const float*)E, ids, d, vocab, (float*)out);
  else
    hipLaunchKernelGGL(k_embed<bf16>, dim3(n), dim3(256), 0, s, (const bf16*)E, ids, d, vocab, (bf16*)out);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_ingest(const T* __restrict__ x, size_t n, float* __restrict__ h) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    h[i] = ld<T>(x, i);
}

// Token i of a pass belongs to segment s (off[s] <= i < off[s+1]) and comes from
// input token src[s] + (i - off[s]).
template <typename T>
__global__ __launch_bounds__(256) void k_ingest_segs(const T* __restrict__ x, const int32_t* __restrict__ off,
                                                     const int32_t* __restrict__ src, int n_seg, int d,
                                                     float* __restrict__ h) {
  const int i = blockIdx.x;
  int lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const size_t from = (size_t)(src[lo] + (i - off[lo])) * d, to = (size_t)i * d;
  for (int e = threadIdx.x; e < d; e += blockDim.x) h[to + e] = ld<T>(x, from + e);
}

hipError_t ingest_segs(int st, const void* x, Segs sg, const int32_t* src, int d, float* h, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  if (st == DT_F32)
    hipLaunchKernelGGL(k_ingest_segs<float>, dim3(sg.n_tok), dim3(256), 0, s, (const float*)x, sg.off, src, sg.n_seg,
                       d, h);
  else
    hipLaunchKernelGGL(k_ingest_segs<bf16>, dim3(sg.n_tok), dim3(256), 0, s, (const bf16*)x, sg.off, src, sg.n_seg,
                       d, h);
  return hipGetLastError();
}

hipError_t ingest(int st, const void* x, int n, int d, float* h, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const size_t tot = (size_t)n * d;
  const int blocks = (int)((tot + 255) / 256 < 65536 ? (tot + 255) / 256 : 65536);
  if (st == DT_F32)
    hipLaunchKernelGGL(k_ingest<float>, dim3(blocks), dim3(256), 0, s, (const float*)x, tot, h);
  else
    hipLaunchKernelGGL(k_ingest<bf16>, dim3(blocks), dim3(256), 0, s, (const bf16*)x, tot, h);
  return hipGetLastError();
}

template <typename TS, typename TC>
__global__ __launch_bounds__(256) void k_pack_gu(const TS* __restrict__ gate, const TS* __restrict__ up,
                                                 const float* __restrict__ gain, int d, TC* __restrict__ dst) {
  const int r = blockIdx.x;  // packed row
  const int blk = r / (2 * GU_BLOCK), j = r % (2 * GU_BLOCK);
  const TS* src = j < GU_BLOCK ? gate + (size_t)(blk * GU_BLOCK + j) * d
                               : up + (size_t)(blk * GU_BLOCK + j - GU_BLOCK) * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) st<TC>(dst, (size_t)r * d + i, ld<TS>(src, i) * gain[i]);
}

hipError_t pack_gate_up(int st_, int ct, const void* gate, const void* up, const float* gain, int F, int d, void* dst,
                        hipStream_t s) {
  if (st_ == DT_F32 && ct == DT_F32)
    hipLaunchKernelGGL((k_pack_gu<float, float>), dim3(2 * F), dim3(256), 0, s, (const float*)gate,
                       (const float*)up, gain, d, (float*)dst);
  else if (st_ == DT_BF16 && ct == DT_F16)
    hipLaunchKernelGGL((k_pack_gu<bf16, f16>), dim3(2 * F), dim3(256), 0, s, (const bf16*)gate, (const bf16*)up,
                       gain, d, (f16*)dst);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename TS, typename TC>
__global__ __launch_bounds__(256) void k_convert(const TS* __restrict__ src, size_t rows, int cols,
                                                 const float* __restrict__ gain, TC* __restrict__ dst) {
  const size_t n = rows * (size_t)cols;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    st<TC>(dst, i, gain ? ld<TS>(src, i) * gain[i % cols] : ld<TS>(src, i));
}

hipError_t convert(int st_, int ct, const void* src, size_t rows, int cols, const float* gain, void* dst,
                   hipStream_t s) {
  const size_t n = rows * (size_t)cols;
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 65536 ? (n + 255) / 256 : 65536);
  if (st_ == DT_F32 && ct == DT_F32)
    hipLaunchKernelGGL((k_convert<float, float>), dim3(blocks), dim3(256), 0, s, (const float*)src, rows, cols, gain,
                       (float*)dst);
  else if (st_ == DT_BF16 && ct == DT_F16)
    hipLaunchKernelGGL((k_convert<bf16, f16>), dim3(blocks), dim3(256), 0, s, (const bf16*)src, rows, cols, gain,
                       (f16*)dst);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

__global__ void k_rope_table(float2* tab, int cap, int half, double log2_theta_over_dh2) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= cap * half) return;
  const int t = idx / half, i = idx % half;
  // theta^(-2i/dh) = 2^(-i * log2(theta) * 2/dh)
  const double ang = (double)t * exp2(-(double)i * log2_theta_over_dh2);
  double sn, cs;
  sincos(ang, &sn, &cs);
  tab[idx] = make_float2((float)cs, (float)sn);
}

hipError_t rope_table(float2* tab, int cap, int dh, float theta, hipStream_t s) {
  const int half = dh / 2;
  const double l = 2.0 * log2((double)theta) / (double)dh;
  hipLaunchKernelGGL(k_rope_table, dim3((cap * half + 255) / 256), dim3(256), 0, s, tab, cap, half, l);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_gather_last(const float* __restrict__ h, const int32_t* __restrict__ row,
                                                     const int32_t* __restrict__ off, int d,
                                                     float* __restrict__ h_last, f16* __restrict__ h_last16,
                                                     f16* __restrict__ h_last16lo) {
  const int sidx = blockIdx.x;
  const int last = off[sidx + 1] - 1;
  const float* src = h + (size_t)last * d;
  const size_t o = (size_t)row[sidx] * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = src[i];
    h_last[o + i] = v;
    if (h_last16) split16(v, h_last16, h_last16lo, o + i);
  }
}

hipError_t gather_last(const float* h, Segs sg, int d, float* h_last, hipStream_t s, void* h_last16,
                       void* h_last16lo) {
  if (sg.n_seg <= 0) return hipSuccess;
  if (h_last16lo && !h_last16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gather_last, dim3(sg.n_seg), dim3(256), 0, s, h, sg.row, sg.off, d, h_last, (f16*)h_last16,
                     (f16*)h_last16lo);
  return hipGetLastError();
}

__global__ void k_update_lens(int32_t* lens, const int32_t* add, int B, int set) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    const int32_t a = add[b];
    lens[b] = set ? (a > 0 ? a : lens[b]) : lens[b] + a;  // set: rows with no tokens keep their length
  }
}

hipError_t update_lens(int32_t* lens, const int32_t* add, int B, int set, hipStream_t s) {
  hipLaunchKernelGGL(k_update_lens, dim3((B + 255) / 256), dim3(256), 0, s, lens, add, B, set);
  return hipGetLastError();
}

// rank of row t = rows strictly longer + rows as long with a lower index
__global__ void k_len_order(const int32_t* __restrict__ lens, int B, int32_t* __restrict__ order) {
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < B; t += gridDim.x * blockDim.x) {
    const int lt = lens[t];
    int r = 0;
    for (int j = 0; j < B; ++j) {
      const int lj = lens[j];
      r += (lj > lt) | ((lj == lt) & (j < t));
    }
    order[r] = t;
  }
}

hipError_t len_order(const int32_t* lens, int B, int32_t* order, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_len_order, dim3((B + 255) / 256), dim3(256), 0, s, lens, B, order);
  return hipGetLastError();
}

}  // namespace ams

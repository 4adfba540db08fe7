// Projection and feed-forward GEMMs: y = u W^T with fused epilogues.
//
//  * k_gemm_skinny  (fp16, M <= 64 tokens: the per-action decode pass).  HBM
//    bound on the weights: every weight byte is read exactly once.  A
//    workgroup owns a strip of 16 (or 32 for SwiGLU) packed weight rows; its
//    waves split K in chunks of 128 and run v_mfma_f32_16x16x32_f16 with the
//    weight rows on the M side and up to 64 tokens as 1..4 column blocks, so a
//    weight fragment is loaded once and reused for every token block.  The
//    per-wave partial sums meet in LDS; the epilogue (store / residual add /
//    SiLU-gate) runs on the reduced values.  Up to 16 tokens it can also
//    apply the preceding RMSNorm itself (gemv_rmsnorm).  RMSNorm gains are
//    folded into the packed weights, so every GEMM consumes h / rms(h).
//  * k_gemm_tiled   (fp16, M > 64: prefix build and observation extension).
//    128x128x64 tiles, 4 waves each owning 64x64 as 4x4 MFMA 16x16x32 blocks,
//    LDS double buffering with one barrier per K step, epilogue staged
//    through LDS so global stores are row-contiguous.
//  * k_gemm_f32     (fp32 model dtype): 64x64x16 FMA tiles, same epilogue.
#include "common.h"
#include "kernels.h"

namespace ams {

__device__ __forceinline__ half8 as_half8(uint4 v) { return __builtin_bit_cast(half8, v); }

// ----------------------------------------------------------------------------
// skinny: M <= 64
//
// Each wave requests the weight and activation fragments of up to CPW of its
// K chunks before the first MFMA, so its loads overlap in one round trip; a
// residual epilogue's h values are requested at kernel entry for the same
// reason.  The K range a wave covers is rotated by the workgroup index, so
// concurrent workgroups read different parts of the shared activations.
//
// NRM (M <= 16): the input is the fp16 copy of the residual stream h [M][K]
// and the kernel applies RMSNorm itself: the MFMA consumes it as is, the sum
// of squares of each token row comes from the same fragments (reduced across
// the waves, which together cover all of K), and the 1/rms scale multiplies
// the result in the epilogue.  The RMSNorm gain is folded into W at packing.
//
// RESID may also write an fp16 copy of the updated residual rows (out16, same
// leading dimension), the input of the next fused-RMSNorm GEMV.

template <int RB, int MB, int EPI, bool NRM>
__global__ __launch_bounds__(512) void k_gemm_skinny(const f16* __restrict__ xin, float eps,
                                                     const f16* __restrict__ W, int M, int K,
                                                     void* __restrict__ out, int ldo, f16* __restrict__ out16) {
  static_assert(!NRM || MB == 1, "the fused RMSNorm handles up to 16 tokens");
  extern __shared__ float red[];  // [nw][RB][MB][64 lanes][4], then (NRM) wsum[<=16 waves][16] + rstd[16]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * (RB * 16);
  const int nchunks = K >> 7;
  const int wk = (wave + blockIdx.x) % nw;
  const int c0 = wk * nchunks / nw, c1 = (wk + 1) * nchunks / nw;

  f32x4 acc[RB][MB];
#pragma unroll
  for (int a = 0; a < RB; ++a)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const f16* wrow[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) wrow[rb] = W + (size_t)(n0 + rb * 16 + r) * K + g * 8;
  bool uok[MB];
  const f16* urow[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int tok = mb * 16 + r;
    uok[mb] = tok < M;
    urow[mb] = xin + (size_t)(uok[mb] ? tok : 0) * K + g * 8;
  }
  float ss = 0.f;  // NRM: this lane's share of sum(h^2) of token r

  // the residual epilogue's h values do not depend on this kernel: request them first
  constexpr int EPT = (MB * 256 + 63) / 64;  // epilogue values per thread at the smallest workgroup
  float hres[EPI == EPI_RESID ? RB * EPT : 1];
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int idx = threadIdx.x + e * blockDim.x;
      const int mb = idx >> 8, ln = (idx >> 2) & 63, i = idx & 3;
      const int tok = mb * 16 + (ln & 15), row = 4 * (ln >> 4) + i;
      const bool ok = idx < MB * 256 && tok < M;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        hres[rb * EPT + e] = ok ? ((const float*)out)[(size_t)tok * ldo + n0 + rb * 16 + row] : 0.f;
    }
  }

  // chunks in flight per wave: up to CPW loads are issued before the first MFMA
  constexpr int CPW = RB + MB <= 2 ? 4 : 2;
  uint4 fw[CPW][RB][4], fu[CPW][MB][4];
  for (int cb = c0; cb < c1; cb += CPW) {
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      if (cb + j < c1) {
        const int kb = (cb + j) << 7;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) fw[j][rb][i] = *(const uint4*)(wrow[rb] + kb + 32 * i);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            fu[j][mb][i] = uok[mb] ? *(const uint4*)(urow[mb] + kb + 32 * i) : uint4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      if (cb + j < c1) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const half8 v = as_half8(fu[j][mb][i]);
            if constexpr (NRM) {
#pragma unroll
              for (int e = 0; e < 8; ++e) ss = fmaf((float)v[e], (float)v[e], ss);
            }
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
              acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(fw[j][rb][i]), v, acc[rb][mb], 0, 0, 0);
          }
      }
    }
  }

#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[(((wave * RB + rb) * MB + mb) * 64 + lane) * 4 + i] = acc[rb][mb][i];
  float* rstd = red + (size_t)nw * RB * MB * 256 + 256;
  if constexpr (NRM) {
    float* wsum = rstd - 256;  // [16 waves][16 tokens]
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    if (lane < 16) wsum[wave * 16 + lane] = ss;
    __syncthreads();
    if (threadIdx.x < 16) {
      float t = 0.f;
      for (int w = 0; w < nw; ++w) t += wsum[w * 16 + threadIdx.x];
      rstd[threadIdx.x] = 1.0f / sqrtf(t / (float)K + eps);
    }
  }
  __syncthreads();

  // value (rb, mb, ln, i) is packed row n0 + rb*16 + 4*(ln>>4) + i, token mb*16 + (ln&15)
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int idx = threadIdx.x + e * blockDim.x;
    if (idx >= MB * 256) break;
    const int mb = idx >> 8, ln = (idx >> 2) & 63, i = idx & 3;
    const int tok = mb * 16 + (ln & 15);
    if (tok >= M) continue;
    const int row = 4 * (ln >> 4) + i;
    float v[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float t = 0.f;
      for (int w = 0; w < nw; ++w) t += red[(((w * RB + rb) * MB + mb) * 64 + ln) * 4 + i];
      if constexpr (NRM) t *= rstd[tok];
      v[rb] = t;
    }
    if constexpr (EPI == EPI_STORE) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) ((float*)out)[(size_t)tok * ldo + n0 + rb * 16 + row] = v[rb];
    } else if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const size_t o = (size_t)tok * ldo + n0 + rb * 16 + row;
        const float hn = hres[rb * EPT + e] + v[rb];
        ((float*)out)[o] = hn;
        if (out16) st<f16>(out16, o, hn);
      }
    } else {
      st<f16>((f16*)out, (size_t)tok * ldo + (n0 >> 1) + row, silu(v[0]) * v[RB - 1]);
    }
  }
}

template <int RB, int MB, int EPI, bool NRM>
static hipError_t launch_skinny(const f16* x, float eps, const f16* W, int M, int N, int K, void* out, int ldo,
                                f16* out16, hipStream_t s) {
  const int nchunks = K >> 7;
  int nw = 8;  // <= 512 threads: leaves 256 VGPRs for the chunks in flight
  while (nw > 1 && nw * RB * MB * 1024 > 65536) nw >>= 1;
  while (nw > 1 && nw > nchunks) nw >>= 1;
  const size_t lds = (size_t)nw * RB * MB * 1024 + (NRM ? (256 + 16) * 4 : 0);
  hipLaunchKernelGGL((k_gemm_skinny<RB, MB, EPI, NRM>), dim3(N / (RB * 16)), dim3(64 * nw), lds, s, x, eps, W, M,
                     K, out, ldo, out16);
  return hipGetLastError();
}

template <int EPI>
static hipError_t skinny_mb(const f16* u, const f16* W, int M, int N, int K, void* out, int ldo, f16* out16,
                            hipStream_t s) {
  constexpr int RB = EPI == EPI_SWIGLU ? 2 : 1;
  if (M <= 16) return launch_skinny<RB, 1, EPI, false>(u, 0.f, W, M, N, K, out, ldo, out16, s);
  if (M <= 32) return launch_skinny<RB, 2, EPI, false>(u, 0.f, W, M, N, K, out, ldo, out16, s);
  if (M <= 48) return launch_skinny<RB, 3, EPI, false>(u, 0.f, W, M, N, K, out, ldo, out16, s);
  return launch_skinny<RB, 4, EPI, false>(u, 0.f, W, M, N, K, out, ldo, out16, s);
}

// ----------------------------------------------------------------------------
// shared epilogue for tiles staged in LDS as Cs[BM][BN + 4] (fp32)

template <int EPI, typename TO, int BM, int BN>
__device__ __forceinline__ void tile_epilogue(const float* Cs, int m0, int n0, int M, void* out, int ldo) {
  constexpr int LDC = BN + 4;
  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int OC = BN / 2;
    for (int idx = threadIdx.x; idx < BM * OC; idx += blockDim.x) {
      const int rr = idx / OC, c = idx % OC;
      if (m0 + rr >= M) continue;
      const int blk = c / GU_BLOCK, j = c % GU_BLOCK;
      const float gt = Cs[rr * LDC + blk * 2 * GU_BLOCK + j];
      const float up = Cs[rr * LDC + blk * 2 * GU_BLOCK + GU_BLOCK + j];
      st<TO>((TO*)out, (size_t)(m0 + rr) * ldo + (n0 >> 1) + c, silu(gt) * up);
    }
  } else {
    for (int idx = threadIdx.x; idx < BM * BN; idx += blockDim.x) {
      const int rr = idx / BN, c = idx % BN;
      if (m0 + rr >= M) continue;
      float* p = (float*)out + (size_t)(m0 + rr) * ldo + n0 + c;
      if constexpr (EPI == EPI_STORE) *p = Cs[rr * LDC + c];
      else *p += Cs[rr * LDC + c];
    }
  }
}

// ----------------------------------------------------------------------------
// tiled f16 MFMA: M > 64

constexpr int TBM = 128, TBN = 128, TBK = 64, TLDK = TBK + 8;
constexpr int T_AB_BYTES = 2 * 2 * TBM * TLDK * 2;  // double-buffered A and B tiles (fp16)
constexpr int T_C_BYTES = TBM * (TBN + 4) * 4;      // fp32 staging for the epilogue
constexpr int T_LDS = T_AB_BYTES > T_C_BYTES ? T_AB_BYTES : T_C_BYTES;

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_tiled(const f16* __restrict__ u, const f16* __restrict__ W,
                                                    int M, int K, void* __restrict__ out, int ldo) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[T_LDS];
  f16* As = (f16*)smem;                  // [2][TBM][TLDK]
  f16* Bs = As + 2 * TBM * TLDK;          // [2][TBN][TLDK]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * TBM, n0 = blockIdx.x * TBN;

  // global -> register mapping: thread loads 32 consecutive k of one row of A and of B
  const int lrow = tid >> 1, lk = (tid & 1) * 32;
  const bool arow_ok = m0 + lrow < M;
  const f16* ag = u + (size_t)(arow_ok ? m0 + lrow : 0) * K + lk;
  const f16* bg = W + (size_t)(n0 + lrow) * K + lk;

  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
#define AMS_GLOAD(k0)                                                                  \
  do {                                                                                 \
    const uint4 z = {0u, 0u, 0u, 0u};                                                  \
    ra0 = arow_ok ? *(const uint4*)(ag + (k0)) : z;                                    \
    ra1 = arow_ok ? *(const uint4*)(ag + (k0) + 8) : z;                                \
    ra2 = arow_ok ? *(const uint4*)(ag + (k0) + 16) : z;                               \
    ra3 = arow_ok ? *(const uint4*)(ag + (k0) + 24) : z;                               \
    rb0 = *(const uint4*)(bg + (k0));                                                  \
    rb1 = *(const uint4*)(bg + (k0) + 8);                                              \
    rb2 = *(const uint4*)(bg + (k0) + 16);                                             \
    rb3 = *(const uint4*)(bg + (k0) + 24);                                             \
  } while (0)
#define AMS_LSTORE(buf)                                                                \
  do {                                                                                 \
    uint4* a_ = (uint4*)(As + ((buf) * TBM + lrow) * TLDK + lk);                       \
    uint4* b_ = (uint4*)(Bs + ((buf) * TBN + lrow) * TLDK + lk);                       \
    a_[0] = ra0; a_[1] = ra1; a_[2] = ra2; a_[3] = ra3;                                \
    b_[0] = rb0; b_[1] = rb1; b_[2] = rb2; b_[3] = rb3;                                \
  } while (0)

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = K / TBK;
  AMS_GLOAD(0);
  AMS_LSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) AMS_GLOAD((kt + 1) * TBK);
#pragma unroll
    for (int ks = 0; ks < TBK / 32; ++ks) {
      half8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *(const half8*)(As + (cur * TBM + wm * 64 + i * 16 + r) * TLDK + ks * 32 + g * 8);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *(const half8*)(Bs + (cur * TBN + wn * 64 + j * 16 + r) * TLDK + ks * 32 + g * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) AMS_LSTORE(cur ^ 1);
    __syncthreads();
  }
#undef AMS_GLOAD
#undef AMS_LSTORE

  // C block (i, j): lane holds rows 4g..4g+3 (tokens) of column r (weight row)
  float* Cs = (float*)smem;
  constexpr int LDC = TBN + 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Cs[(wm * 64 + i * 16 + 4 * g + e) * LDC + wn * 64 + j * 16 + r] = acc[i][j][e];
  __syncthreads();
  tile_epilogue<EPI, f16, TBM, TBN>(Cs, m0, n0, M, out, ldo);
}

// ----------------------------------------------------------------------------
// fp32 model dtype

constexpr int FBM = 64, FBN = 64, FBK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ u, const float* __restrict__ W,
                                                  int M, int K, void* __restrict__ out, int ldo) {
  constexpr int LDC = FBN + 4;
  __shared__ float As[FBK][FBM + 4], Bs[FBK][FBN + 4];
  __shared__ float Cs[FBM * LDC];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * FBM, n0 = blockIdx.x * FBN;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FBK) {
    for (int idx = tid; idx < FBM * FBK; idx += 256) {
      const int rr = idx / FBK, kk = idx % FBK;
      As[kk][rr] = (m0 + rr < M) ? u[(size_t)(m0 + rr) * K + k0 + kk] : 0.f;
      Bs[kk][rr] = W[(size_t)(n0 + rr) * K + k0 + kk];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FBK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) Cs[(ty * 4 + i) * LDC + tx * 4 + j] = acc[i][j];
  __syncthreads();
  tile_epilogue<EPI, float, FBM, FBN>(Cs, m0, n0, M, out, ldo);
}

// ----------------------------------------------------------------------------

template <int EPI>
static hipError_t gemm_epi(int ct, const void* u, const void* W, int M, int N, int K, void* out, int ldo,
                           void* out16, hipStream_t s) {
  // the fp16 residual copy is produced by the decode GEMV only
  if (out16 && (EPI != EPI_RESID || ct != DT_F16 || M > 64)) return hipErrorInvalidValue;
  if (ct == DT_F32) {
    hipLaunchKernelGGL((k_gemm_f32<EPI>), dim3(N / FBN, (M + FBM - 1) / FBM), dim3(256), 0, s,
                       (const float*)u, (const float*)W, M, K, out, ldo);
    return hipGetLastError();
  }
  if (M <= 64) return skinny_mb<EPI>((const f16*)u, (const f16*)W, M, N, K, out, ldo, (f16*)out16, s);
  hipLaunchKernelGGL((k_gemm_tiled<EPI>), dim3(N / TBN, (M + TBM - 1) / TBM), dim3(256), 0, s,
                     (const f16*)u, (const f16*)W, M, K, out, ldo);
  return hipGetLastError();
}

hipError_t gemm(int ct, int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo,
                hipStream_t s, void* out16) {
  if (M <= 0) return hipSuccess;
  switch (epi) {
    case EPI_STORE: return gemm_epi<EPI_STORE>(ct, u, W, M, N, K, out, ldo, out16, s);
    case EPI_RESID: return gemm_epi<EPI_RESID>(ct, u, W, M, N, K, out, ldo, out16, s);
    default: return gemm_epi<EPI_SWIGLU>(ct, u, W, M, N, K, out, ldo, out16, s);
  }
}

hipError_t gemv_rmsnorm(int ct, int epi, const void* h16, float eps, const void* W, int M, int N, int K, void* out,
                        int ldo, hipStream_t s, void* out16) {
  if (M <= 0) return hipSuccess;
  if (ct != DT_F16 || M > 16) return hipErrorInvalidValue;
  if (out16 && epi != EPI_RESID) return hipErrorInvalidValue;
  const f16* x = (const f16*)h16;
  const f16* w = (const f16*)W;
  switch (epi) {
    case EPI_STORE: return launch_skinny<1, 1, EPI_STORE, true>(x, eps, w, M, N, K, out, ldo, nullptr, s);
    case EPI_RESID: return launch_skinny<1, 1, EPI_RESID, true>(x, eps, w, M, N, K, out, ldo, (f16*)out16, s);
    default: return launch_skinny<2, 1, EPI_SWIGLU, true>(x, eps, w, M, N, K, out, ldo, nullptr, s);
  }
}

}  // namespace ams

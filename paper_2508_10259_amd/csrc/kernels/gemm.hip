// Projection and feed-forward GEMMs: y = u W^T with fused epilogues.
//
//  * k_gemm_skinny  (fp16, M <= 64 tokens: the per-action decode pass).  HBM
//    bound on the weights: every weight byte is read exactly once.  A
//    workgroup owns a strip of 16 (or 32 for SwiGLU: 16 gate + 16 up) packed weight rows; its
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
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace ams {

__device__ __forceinline__ half8 as_half8(uint4 v) { return __builtin_bit_cast(half8, v); }
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// ----------------------------------------------------------------------------
// skinny: M <= 64
//
// Each wave requests the weight and activation fragments of up to CPW of its
// K chunks before the first MFMA, so its loads overlap in one round trip; a
// residual epilogue's h values are requested at kernel entry for the same
// reason.  The K range a wave covers is rotated by the workgroup index, so
// concurrent workgroups read different parts of the shared activations.
//
// Compensated input (LO != 0): the activations arrive as an fp16 pair
// x = hi + lo (lo = the rounding error of hi), and W x = W hi + W lo, so the
// product carries about 22 significant bits of x instead of 11.  With up to 8
// tokens (LO == 1) the pair shares one MFMA: B columns 0..7 take hi, columns
// 8..15 take lo of the same tokens, and the epilogue adds the two halves;
// otherwise (LO == 2) lo has its own fragments and MFMAs.
//
// NRM (M <= 16): the input is the (fp16 or fp16-pair) copy of the residual
// stream h [M][K] and the kernel applies RMSNorm itself: the MFMA consumes it
// as is, the sum of squares of each token row comes from the hi fragments
// (reduced across the waves, which together cover all of K), and the 1/rms
// scale multiplies the result in the epilogue.  The RMSNorm gain is folded
// into W at packing.  Taking the statistic from hi alone changes it by about
// 2^-11 / sqrt(K) relative for rounding errors of random sign (the product,
// where one term's error does not average out, takes hi + lo).
//
// RESID may also write the updated residual rows as fp16 (ohi, and olo for
// the pair), the input of the next fused-RMSNorm GEMV; SWIGLU may write the
// rounding error of its fp16 output to olo.

struct SkinnyArgs {
  const f16* xhi;  // [M][K]
  const f16* xlo;  // [M][K] or NULL
  float eps;
  const f16* W;    // [N][K]
  int M, K;
  void* out;
  int ldo;
  f16* ohi;  // RESID only, or NULL
  f16* olo;  // RESID / SWIGLU, or NULL
};

// most waves per workgroup: 16 for the SwiGLU strip with one token block (its
// two chunks in flight fit 128 VGPRs), 8 otherwise (256 VGPRs)
template <int RB, int MB, int LO>
constexpr int skinny_max_waves() {
  return RB == 2 && MB == 1 && LO != 2 ? 16 : 8;
}

template <int RB, int MB, int LO>
constexpr int skinny_cpw() {
  return (RB + MB * (LO == 2 ? 2 : 1)) <= 2 ? 4 : ((RB + MB * (LO == 2 ? 2 : 1)) <= 4 ? 2 : 1);
}

template <int RB, int MB, int EPI, bool NRM, int LO>
__global__ __launch_bounds__((64 * skinny_max_waves<RB, MB, LO>())) void k_gemm_skinny(SkinnyArgs a) {
  static_assert(!NRM || MB == 1, "the fused RMSNorm handles up to 16 tokens");
  static_assert(!NRM || EPI != EPI_PART, "the RMS statistic needs all of K");
  static_assert(LO != 1 || MB == 1, "the packed pair handles up to 8 tokens");
  constexpr int LB = LO == 2 ? MB : 1;  // lo fragment blocks (unused unless LO == 2)
  extern __shared__ float red[];  // [nw][RB][MB][64 lanes][4], then (NRM) wsum[<=16 waves][16] + rstd[16]
  const int lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: chunk loops branch on scalars
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * (RB * 16);
  const int M = a.M, K = a.K, ldo = a.ldo;
  // K chunks of this workgroup: split blockIdx.y of gridDim.y (EPI_PART), shared by the waves
  const int nchunks = K >> 7, S = gridDim.y, sp = blockIdx.y;
  const int s0 = sp * nchunks / S, s1 = (sp + 1) * nchunks / S;
  const int wk = (wave + blockIdx.x) % nw;
  const int c0 = s0 + wk * (s1 - s0) / nw, c1 = s0 + (wk + 1) * (s1 - s0) / nw;

  f32x4 acc[RB][MB];
#pragma unroll
  for (int q = 0; q < RB; ++q)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[q][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const f16* wrow[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) wrow[rb] = a.W + (size_t)(n0 + rb * 16 + r) * K + g * 8;
  // B-operand rows of this lane: token mb*16 + r (LO == 1: token r & 7, hi for r < 8, lo above).
  // Columns of tokens >= M read token 0 instead of being masked (a masked load
  // costs a branch per load): they only feed output columns that are never
  // stored, and statistics that are never read.
  const f16* urow[MB];
  const f16* lrow[LB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int tok = LO == 1 ? (r & 7) : mb * 16 + r;
    const size_t off = (size_t)(tok < M ? tok : 0) * K + g * 8;
    urow[mb] = (LO == 1 && r >= 8 ? a.xlo : a.xhi) + off;
    if constexpr (LO == 2) lrow[mb] = a.xlo + off;
  }
  float ss0 = 0.f, ss1 = 0.f;  // NRM: this lane's share of sum(x^2) of its token (two chains)

  // the residual epilogue's h values do not depend on this kernel: request them first
  constexpr int EPT = (MB * 256 + 63) / 64;  // epilogue values per thread at the smallest workgroup
  float hres[EPI == EPI_RESID ? RB * EPT : 1];
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int idx = threadIdx.x + e * blockDim.x;
      const int mb = idx >> 8, ln = (idx >> 2) & 63, i = idx & 3;
      const int tok = mb * 16 + (ln & 15), row = 4 * (ln >> 4) + i;
      const bool ok = idx < MB * 256 && tok < M && (LO != 1 || (ln & 15) < 8);
      const size_t at = (size_t)(ok ? tok : 0) * ldo + n0 + row;  // unused values read row 0
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) hres[rb * EPT + e] = ((const float*)a.out)[at + rb * 16];
    }
  }

  // chunks in flight per wave: up to CPW loads are issued before the first MFMA
  constexpr int CPW = skinny_cpw<RB, MB, LO>();
  uint4 fw[CPW][RB][4], fu[CPW][MB][4], fl[CPW][LB][4];
  for (int cb = c0; cb < c1; cb += CPW) {
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      if (cb + j < c1) {
        const int kb = (cb + j) << 7;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) fw[j][rb][i] = ld_stream(wrow[rb] + kb + 32 * i);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            fu[j][mb][i] = *(const uint4*)(urow[mb] + kb + 32 * i);
            if constexpr (LO == 2) fl[j][mb][i] = *(const uint4*)(lrow[mb] + kb + 32 * i);
          }
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
            if constexpr (NRM) {  // the statistic reads hi only (LO == 1: lanes r >= 8 are unused)
              const half2v* p2 = (const half2v*)&fu[j][mb][i];
              ss0 = __builtin_amdgcn_fdot2(p2[0], p2[0], ss0, false);
              ss1 = __builtin_amdgcn_fdot2(p2[1], p2[1], ss1, false);
              ss0 = __builtin_amdgcn_fdot2(p2[2], p2[2], ss0, false);
              ss1 = __builtin_amdgcn_fdot2(p2[3], p2[3], ss1, false);
            }
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
              acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(fw[j][rb][i]), v, acc[rb][mb], 0, 0, 0);
              if constexpr (LO == 2)
                acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(fw[j][rb][i]), as_half8(fl[j][mb][i]),
                                                                      acc[rb][mb], 0, 0, 0);
            }
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
    float ss = ss0 + ss1;
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    if (lane < 16) wsum[wave * 16 + lane] = ss;
    __syncthreads();
    if (threadIdx.x < 16) {
      float t = 0.f;
      for (int w = 0; w < nw; ++w) t += wsum[w * 16 + threadIdx.x];
      rstd[threadIdx.x] = 1.0f / sqrtf(t / (float)K + a.eps);
    }
  }
  __syncthreads();

  // value (rb, mb, ln, i) is packed row n0 + rb*16 + 4*(ln>>4) + i, B column mb*16 + (ln&15);
  // summed over the waves (and, LO == 1, over the hi and lo columns ln and ln+8)
  auto reduced = [&](int rb, int mb, int ln, int i) {
    float t = 0.f;
    for (int w = 0; w < nw; ++w) {
      t += red[(((w * RB + rb) * MB + mb) * 64 + ln) * 4 + i];
      if constexpr (LO == 1) t += red[(((w * RB + rb) * MB + mb) * 64 + ln + 8) * 4 + i];
    }
    return t;
  };
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int idx = threadIdx.x + e * blockDim.x;
    if (idx >= MB * 256) break;
    const int mb = idx >> 8, ln = (idx >> 2) & 63, i = idx & 3;
    const int tok = mb * 16 + (ln & 15);
    if (tok >= M || (LO == 1 && (ln & 15) >= 8)) continue;
    const int row = 4 * (ln >> 4) + i;
    const float sc = NRM ? rstd[tok] : 1.f;
    if constexpr (EPI == EPI_STORE) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        ((float*)a.out)[(size_t)tok * ldo + n0 + rb * 16 + row] = reduced(rb, mb, ln, i) * sc;
    } else if constexpr (EPI == EPI_PART) {  // this split's partial sums: out[sp][tok][n]
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        ((float*)a.out)[((size_t)sp * M + tok) * ldo + n0 + rb * 16 + row] = reduced(rb, mb, ln, i);
    } else if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const size_t o = (size_t)tok * ldo + n0 + rb * 16 + row;
        const float hn = hres[rb * EPT + e] + reduced(rb, mb, ln, i) * sc;
        ((float*)a.out)[o] = hn;
        if (a.ohi) split16(hn, a.ohi, a.olo, o);
      }
    } else {  // the strip's first 16 rows are gate rows, the next 16 the up rows of the same outputs
      const float gt = reduced(0, mb, ln, i) * sc, up = reduced(RB - 1, mb, ln, i) * sc;
      split16(silu(gt) * up, (f16*)a.out, a.olo, (size_t)tok * ldo + (n0 >> 1) + row);
    }
  }
}

template <int RB, int MB, int EPI, bool NRM, int LO>
static hipError_t launch_skinny(const SkinnyArgs& a, int N, hipStream_t s, int splits = 1) {
  // waves per workgroup: at most 64 KB of reduction LDS and at least one chunk
  // per wave; the 16-wave variant takes 16 only when every wave then gets a
  // full batch of CPW chunks (all chunks go out in one round), 8 otherwise
  const int nchunks = (a.K >> 7) / splits;
  constexpr int MW = skinny_max_waves<RB, MB, LO>();
  int nw = MW == 16 && nchunks < 16 * skinny_cpw<RB, MB, LO>() ? 8 : MW;
  while (nw > 1 && nw * RB * MB * 1024 > 65536) nw >>= 1;
  while (nw > 1 && nw > nchunks) nw >>= 1;
  const size_t lds = (size_t)nw * RB * MB * 1024 + (NRM ? (256 + 16) * 4 : 0);
  hipLaunchKernelGGL((k_gemm_skinny<RB, MB, EPI, NRM, LO>), dim3(N / (RB * 16), splits), dim3(64 * nw), lds, s, a);
  return hipGetLastError();
}

// token blocks and input form of one skinny launch
template <int EPI, bool NRM>
static hipError_t skinny_dispatch(const SkinnyArgs& a, int N, hipStream_t s) {
  constexpr int RB = EPI == EPI_SWIGLU ? 2 : 1;
  const int M = a.M;
  if (!a.xlo) {
    if (M <= 16) return launch_skinny<RB, 1, EPI, NRM, 0>(a, N, s);
    if constexpr (!NRM) {
      if (M <= 32) return launch_skinny<RB, 2, EPI, false, 0>(a, N, s);
      if (M <= 48) return launch_skinny<RB, 3, EPI, false, 0>(a, N, s);
      return launch_skinny<RB, 4, EPI, false, 0>(a, N, s);
    }
  } else {
    if (M <= 8) return launch_skinny<RB, 1, EPI, NRM, 1>(a, N, s);
    if (M <= 16) return launch_skinny<RB, 1, EPI, NRM, 2>(a, N, s);
    if constexpr (!NRM) {
      if (M <= 32) return launch_skinny<RB, 2, EPI, false, 2>(a, N, s);
      if (M <= 48) return launch_skinny<RB, 3, EPI, false, 2>(a, N, s);
      return launch_skinny<RB, 4, EPI, false, 2>(a, N, s);
    }
  }
  return hipErrorInvalidValue;
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

// Tile rows of TBK + 16 halves (160 bytes): the fragment reads and the staging
// writes (8 lanes fill one row) are free of LDS bank conflicts on gfx950.
constexpr int TBM = 128, TBN = 128, TBK = 64, TLDK = TBK + 16;
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

  // global -> register mapping: thread loads the 16-byte k chunk tid & 7 of rows
  // tid / 8 + 32 q (q < 4) of A and of B
  const int lrow = tid >> 3, lk = (tid & 7) * 8;
  bool aok[4];
  const f16* ag[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    aok[q] = m0 + lrow + 32 * q < M;
    ag[q] = u + (size_t)(aok[q] ? m0 + lrow + 32 * q : 0) * K + lk;
  }
  const f16* bg = W + (size_t)(n0 + lrow) * K + lk;

  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
#define AMS_GLOAD(k0)                                                                  \
  do {                                                                                 \
    const uint4 z = {0u, 0u, 0u, 0u};                                                  \
    ra0 = aok[0] ? *(const uint4*)(ag[0] + (k0)) : z;                                  \
    ra1 = aok[1] ? *(const uint4*)(ag[1] + (k0)) : z;                                  \
    ra2 = aok[2] ? *(const uint4*)(ag[2] + (k0)) : z;                                  \
    ra3 = aok[3] ? *(const uint4*)(ag[3] + (k0)) : z;                                  \
    rb0 = *(const uint4*)(bg + (k0));                                                  \
    rb1 = *(const uint4*)(bg + (size_t)32 * K + (k0));                                 \
    rb2 = *(const uint4*)(bg + (size_t)64 * K + (k0));                                 \
    rb3 = *(const uint4*)(bg + (size_t)96 * K + (k0));                                 \
  } while (0)
#define AMS_LSTORE(buf)                                                                \
  do {                                                                                 \
    f16* a_ = As + ((buf) * TBM + lrow) * TLDK + lk;                                   \
    f16* b_ = Bs + ((buf) * TBN + lrow) * TLDK + lk;                                   \
    *(uint4*)a_ = ra0; *(uint4*)(a_ + 32 * TLDK) = ra1;                                \
    *(uint4*)(a_ + 64 * TLDK) = ra2; *(uint4*)(a_ + 96 * TLDK) = ra3;                  \
    *(uint4*)b_ = rb0; *(uint4*)(b_ + 32 * TLDK) = rb1;                                \
    *(uint4*)(b_ + 64 * TLDK) = rb2; *(uint4*)(b_ + 96 * TLDK) = rb3;                  \
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
// big f16 MFMA tiles: large prefix builds (enough 256 x 256 tiles to fill the chip)
//
// 256 (tokens) x 256 (weight rows) per workgroup, eight waves of 64 x 128
// (4 x 2), K steps of 64 double-buffered in LDS.  The tiles move from global
// memory straight into LDS (global_load_lds_dwordx4: each wave instruction
// fills 1 KB of LDS, lane i the i-th 16 bytes), so no registers stage them.
// A tile row is 128 bytes (8 chunks of 16); chunk c of row R sits in slot
// c ^ (R & 7), which the DMA realises by choosing each lane's source chunk,
// and which keeps the 16-byte fragment reads of 8 consecutive rows on 8
// distinct bank groups.  A wave reuses each A fragment for 8 B fragments and
// each B fragment for 4 A fragments.  The epilogue runs from registers: a lane
// holds 4 consecutive tokens of one weight row per 16 x 16 block, and the gate
// and up blocks of a SwiGLU pair sit side by side in the same lane.  With
// EPI_PART the K steps are cut into gridDim.y splits, each writing its partial
// sums (for medium token counts, where the tiles alone leave CUs idle).

constexpr int GBM = 256, GBN = 256, GBK = 64;
constexpr int G_TILE = 256 * 128;         // bytes of one 256-row A or B tile (rows of 64 fp16)

// LDS of a BN-wide tile pair, double-buffered: [2 stages][A tile | B tile]
template <int BN> constexpr int g_lds() { return 2 * (G_TILE + BN * 128); }

typedef __attribute__((address_space(3))) void* lds_ptr;

// DMA of one K step: wave w moves 1 KB blocks 4w..4w+3 of the A tile and
// BN/64 blocks of the B tile (8 rows each).  Lane i of a block: row R0 + i/8,
// slot i%8, source chunk (i%8) ^ (row & 7).  A rows past the last valid one
// (alast) read it again: they only feed outputs that are never stored.
template <int BN>
__device__ __forceinline__ void big_dma(unsigned char* stage, const f16* A, const f16* B, int K, int k0, int alast,
                                        int wave, int lane) {
  constexpr int BQ = BN / 64;  // B blocks per wave
  const int slot = lane & 7;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int blk = wave * 4 + q;
    const int row = blk * 8 + (lane >> 3);
    const int c = slot ^ (row & 7);
    const int ar = row <= alast ? row : alast;
    __builtin_amdgcn_global_load_lds((const void*)(A + (size_t)ar * K + k0 + c * 8), (lds_ptr)(stage + blk * 1024),
                                     16, 0, 0);
    if (q < BQ) {
      const int bblk = wave * BQ + q;
      const int brow = bblk * 8 + (lane >> 3);
      const int bc = slot ^ (brow & 7);
      __builtin_amdgcn_global_load_lds((const void*)(B + (size_t)brow * K + k0 + bc * 8),
                                       (lds_ptr)(stage + G_TILE + bblk * 1024), 16, 0, 0);
    }
  }
}

// BN = 256, or 192 / 128 for shapes whose 256-wide tiles leave a round of CUs
// mostly idle (QKV of the 1,024-token extension: 192 tiles of 256 x 256 on 256
// CUs, 256 tiles of 256 x 192; the columns past whole rounds of gate|up there
// as 256 x 128 tiles); each wave then covers 64 x BN/2.
template <int EPI, int BN = GBN>
__global__ __launch_bounds__(512) void k_gemm_big(const f16* __restrict__ u, const f16* __restrict__ W, int M,
                                                  int N, int K, void* __restrict__ out, int ldo, KvEpi kv) {
  constexpr int WN = BN / 2, NJ = WN / 16;  // weight rows per wave, 16-row blocks per wave
  constexpr int STAGE = G_TILE + BN * 128;
  static_assert(EPI != EPI_SWIGLU || NJ % 2 == 0, "gate and up blocks come in pairs");
  extern __shared__ __attribute__((aligned(16))) unsigned char gsm[];  // [2 stages][A tile | B tile]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;  // wave tile: tokens wm*64.., weight rows wn*WN..
  // tile order: workgroups are dispatched round-robin over the 8 XCDs, so XCD x
  // (ids = x mod 8) takes a contiguous range of the tile sequence, which walks
  // groups of 8 token tiles down each weight tile: tiles that share a weight
  // (or token) tile run close together on one XCD's L2
  const int tm_n = (M + GBM - 1) / GBM, tn_n = N / BN, T = tm_n * tn_n;
  const int L = blockIdx.x, xcd = L & 7, per = T >> 3, rem = T & 7;
  const int Lx = xcd * per + (xcd < rem ? xcd : rem) + (L >> 3);
  const int grp = Lx / (8 * tn_n), first_m = grp * 8;
  const int gm = tm_n - first_m < 8 ? tm_n - first_m : 8;
  const int in_grp = Lx - grp * 8 * tn_n;
  const int m0 = (first_m + in_grp % gm) * GBM, n0 = (in_grp / gm) * BN;
  const int alast = M - 1 - m0;  // last valid A row of this tile (>= 0)
  // K steps of this workgroup: split blockIdx.y of gridDim.y (EPI_PART; one split otherwise)
  const int KT_all = K / GBK, sp = blockIdx.y, S = gridDim.y;
  const int kt0 = sp * KT_all / S, kt1 = (sp + 1) * KT_all / S;
  const f16* A = u + (size_t)m0 * K + (size_t)kt0 * GBK;
  const f16* B = W + (size_t)n0 * K + (size_t)kt0 * GBK;

  f32x4 acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fragment rows of this lane: A rows wm*64 + 16 i + r, B rows wn*WN + 16 j + r (all = r mod 8)
  const int sw = r & 7;
  const int KT = kt1 - kt0;
  big_dma<BN>(gsm, A, B, K, 0, alast, wave, lane);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    unsigned char* cur = gsm + (kt & 1) * STAGE;
    if (kt + 1 < KT) big_dma<BN>(gsm + ((kt + 1) & 1) * STAGE, A, B, K, (kt + 1) * GBK, alast, wave, lane);
    const unsigned char* Ab = cur + (wm * 64 + r) * 128;
    const unsigned char* Bb = cur + G_TILE + (wn * WN + r) * 128;
    // every fragment of the K step requested in use order, the MFMA groups (8
    // MFMAs: two B fragments times four A fragments) interleaved with the
    // requests of the fragments two groups ahead, so a group does not wait on
    // the LDS round trip of its own operands (on the 7B builds 1.5-2.5% faster
    // than the compiler's order, which requested each group's fragments right
    // before it)
    half8 af[2][4], bfr[2][NJ];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int off = (((4 * ks + g) ^ sw) << 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) af[ks][i] = *(const half8*)(Ab + i * 16 * 128 + off);
#pragma unroll
      for (int j = 0; j < NJ; ++j) bfr[ks][j] = *(const half8*)(Bb + j * 16 * 128 + off);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[ks][i], bfr[ks][j], acc[i][j], 0, 0, 0);
    if constexpr (NJ == 8) {  // sched_group_barrier masks: 0x100 LDS reads, 0x008 MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's DMA into the other stage has landed
    __syncthreads();
  }

  // block (i, j): lane holds tokens tm + 4g + e of weight row tn + r
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tm = m0 + wm * 64 + i * 16 + 4 * g;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int tok = tm + e;
      if (tok >= M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
        // blocks 2p (gate) and 2p+1 (up) of the packed interleave; output column (n >> 1) + r
#pragma unroll
        for (int pr = 0; pr < NJ / 2; ++pr) {
          const int col = ((n0 + wn * WN) >> 1) + pr * 16 + r;
          st<f16>((f16*)out, (size_t)tok * ldo + col, silu(acc[i][2 * pr][e]) * acc[i][2 * pr + 1][e]);
        }
      } else if (EPI == EPI_QKV && n0 + wn * WN >= kv.d) {
        // k or v columns (a wave's 128 columns lie in one of q, k, v: d is a multiple of
        // 256): heads c / dh .. of this wave, written to the token's pool slot as
        // k_kv_append writes them (k rotated by the token's position, rotate-half)
        const int c0 = n0 + wn * WN;
        const bool isk = c0 < 2 * kv.d;
        const size_t base = (size_t)kv.tok_base[tok];
        const int hd0 = (c0 - (isk ? kv.d : 2 * kv.d)) / kv.dh;
        // rotate-half pairs: dims dd and dd + dh/2 of a head are blocks jj and jj + HB/2
        // of its HB = dh/16 blocks (the block index a constant: acc stays in registers)
        auto kstore = [&](auto hbc) __attribute__((always_inline)) {
          constexpr int HB = decltype(hbc)::value;
          const int p = kv.tok_pos[tok], half = HB * 8;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int hh = j / HB, jj = j % HB;  // head of this wave, block within the head
            if (jj < HB / 2) {
              const int dd = 16 * jj + r;  // < half; its partner is dd + half
              const float2 cs = kv.rope[(size_t)p * half + dd];
              const float a = acc[i][j][e], c = acc[i][(j + HB / 2) % NJ][e];
              f16* dst = (f16*)kv.k + base + (size_t)(hd0 + hh) * KV_PAGE * (2 * half);
              st<f16>(dst, dd, a * cs.x - c * cs.y);
              st<f16>(dst, dd + half, a * cs.y + c * cs.x);
            }
          }
        };
        if (isk) {
          if (kv.dh == 128) kstore(std::integral_constant<int, 8>{});
          else kstore(std::integral_constant<int, 4>{});
        } else {
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int col = 16 * j + r, hh = col / kv.dh, dd = col % kv.dh;
            st<f16>((f16*)kv.v + base + (size_t)(hd0 + hh) * KV_PAGE * kv.dh, dd, acc[i][j][e]);
          }
        }
      } else {
        // EPI_PART: this split's partial sums at out[sp][tok][n] (ldo = N)
        const size_t rowo = ((size_t)(EPI == EPI_PART ? sp * M : 0) + tok) * ldo;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          float* p = (float*)out + rowo + n0 + wn * WN + j * 16 + r;
          if constexpr (EPI == EPI_RESID) *p += acc[i][j][e];
          else *p = acc[i][j][e];
        }
      }
    }
  }
}

template <int EPI, int BN = GBN>
static hipError_t launch_big(const f16* u, const f16* W, int M, int N, int K, void* out, int ldo, hipStream_t s,
                             int splits = 1, const KvEpi& kv = KvEpi{}) {
  hipLaunchKernelGGL((k_gemm_big<EPI, BN>), dim3((N / BN) * ((M + GBM - 1) / GBM), splits), dim3(512), g_lds<BN>(),
                     s, u, W, M, N, K, out, ldo, kv);
  return hipGetLastError();
}

// 256 x 256 tile columns that fill whole rounds of the CUs, when the rest
// would leave a last round less than half busy and a round is whole tile
// columns (256 / token tiles an integer); gemm() runs the remaining weight rows
// as 256 x 128 tiles.  At 1,024 tokens the 7B gate|up projection's 344 big
// tiles become 256 (64 columns) + 176 half-width ones for 88 big ones' work.
static int big_main_cols(int M, int N) {
  const int tm = (M + GBM - 1) / GBM, tn = N / GBN;
  if (256 % tm != 0) return tn;
  const int per_round = 256 / tm;
  const int full = tn / per_round * per_round, rest = tn - full;
  if (full == 0 || rest == 0 || 2 * rest * tm > 256) return tn;
  return full;
}

// 256 x 192 tiles when N allows them and they need fewer CU-rounds weighted by
// tile width (rounds of 256 workgroups, one per CU): ceil(T192 / 256) * 192 <
// ceil(T256 / 256) * 256.  At 1,024 tokens the 7B QKV projection takes one
// round of 256 narrower tiles instead of 192 wide ones with 64 CUs idle.
static bool big_narrow(int M, int N) {
  if (N % 192 != 0) return false;
  const long tm = (M + GBM - 1) / GBM;
  const long r256 = (tm * (N / 256) + 255) / 256, r192 = (tm * (N / 192) + 255) / 256;
  return r192 * 192 < r256 * 256;
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

// ----------------------------------------------------------------------------
// wide decode GEMM: 16 < M <= 64 tokens (batched decode), split-K partial sums
//
// A workgroup owns 128 weight rows (8 waves x 16) and one K split.  Every
// 128-wide K chunk of the activations (hi, and lo for the fp16 pair; all M
// tokens) is loaded once per workgroup into double-buffered LDS and read by
// all 8 waves as MFMA B fragments, so activation traffic is about the weight
// traffic instead of M/8 times it; each wave streams its own weight rows into
// registers, WP chunks ahead.  Waves own disjoint rows, so no reduction runs
// at the end: each writes its partial sums, and a reduction kernel applies
// the epilogue (part_store / part_resid / part_swiglu).

// LDS rows of 128 + 16 halves (288 bytes): the MFMA B-fragment reads (lane r
// reads row r, lanes 16 apart the next 16 bytes) are free of bank conflicts at
// that pitch; at 272 bytes every ds_read_b128 took 8 LDS cycles instead of 4.
// Three weight chunks in flight per wave: at 16 rows that fits 80 VGPRs, three
// workgroups per CU, and on the 7B shapes it beat four chunks by 1-5% (QKV at
// 16 rows 23.4 -> 22.1 us, O at 64 rows 15.1 -> 14.4 us; only O at 16 rows lost,
// 9.6 -> 9.9 us); six or eight chunks cost occupancy and were slower.
constexpr int WIDE_ROWS = 128, WIDE_WP = 3, WIDE_LDK = 128 + 16;

// weight fragments of one chunk of a wave's 16 rows from the fragment-ordered
// copy (1 KB of contiguous memory per MFMA step): wstrip = the strip's first
// block + lane * 8.  Measured against row-major loads (each lane 16 bytes of a
// different row) on the 7B shapes: at 64 rows gate|up 51.3 -> 48.8 us, QKV
// 32.6 -> 29.3 us, down 25.6 -> 24.2 us, O 13.2 -> 11.9 us; at 16 rows gate|up
// 38.4 -> 35.2 us, QKV 22.0 -> 20.1 us.
__device__ __forceinline__ void wide_wload_fo(uint4 (&w)[4], const f16* wstrip, int c) {
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = ld_stream(wstrip + ((size_t)c * 4 + i) * 512);
}

// one thread per 16 bytes of the fragment-ordered copy
__global__ __launch_bounds__(256) void k_frag_pack(const f16* __restrict__ W, int N, int K, f16* __restrict__ Wf) {
  const size_t o = (size_t)blockIdx.x * blockDim.x + threadIdx.x;  // 16-byte unit of Wf
  const size_t total = (size_t)N * K / 8;
  if (o >= total) return;
  const int l = (int)(o & 63);
  const size_t blk = o >> 6;  // (s * nch + c) * 4 + i
  const int i = (int)(blk & 3);
  const size_t sc = blk >> 2;
  const int nch = K >> 7;
  const int c = (int)(sc % nch);
  const size_t st = sc / nch;
  const size_t row = st * 16 + (l & 15), col = (size_t)c * 128 + 32 * i + 8 * (l >> 4);
  *(uint4*)(Wf + o * 8) = *(const uint4*)(W + row * K + col);
}

hipError_t frag_pack(const void* W, int N, int K, void* Wf, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (N % 16 != 0 || K % 128 != 0) return hipErrorInvalidValue;
  const size_t units = (size_t)N * K / 8;
  hipLaunchKernelGGL(k_frag_pack, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, s, (const f16*)W, N, K,
                     (f16*)Wf);
  return hipGetLastError();
}

typedef unsigned u32x4v __attribute__((ext_vector_type(4)));
constexpr int WIDE_SC1 = 16;  // cache-policy bits of a buffer access: device scope (sc1)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t wide_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// The reduction of one 128-column tile by the last of its splits to finish
// (EPI_STORE / EPI_SWIGLU / EPI_RESID): every split's partial sums went out
// with device-scope stores, completed before the split counted itself in, so
// the last arrival reads them all (device-scope loads: the XCDs' L2s are not
// coherent with each other) and adds them in split order, the order the
// part_* reductions use.
struct WideEpi {
  unsigned* cnt;        // per-tile arrival counters, zero between launches (the last arrival resets its own)
  void* out;            // STORE: float [M][ldo]; SWIGLU: fp16 [M][ldo] (ldo = N / 2)
  void* olo;            // SWIGLU: rounding error of out (fp16) or NULL
  int ldo;
  float* h;             // RESID: residual [M][N] (+= the product)
  void* o16;            // RESID: fp16 pair of the new rows (o16, olo2) or NULL
  void* olo2;
  float* ss_out;        // RESID: sums of squares of the new rows per 128 columns, [M][N / 128], or NULL
  const float* ss_in;   // STORE / SWIGLU: the sums of squares of the unnormalised input rows, [M][K / 128], or NULL
  float eps;
};

template <int EPI>
__device__ void wide_reduce(const WideEpi& e, __amdgpu_buffer_rsrc_t pr, int S, int M, int N, int K, int n0) {
  __shared__ float rs[64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if constexpr (EPI != EPI_RESID) {  // 1/rms of each input row, as row_rstd computes it
    const int nss = K / 128;
    for (int m = wave; m < M; m += 8) {
      float t = 0.f;
      if (e.ss_in)
        for (int k = lane; k < nss; k += 64) t += e.ss_in[(size_t)m * nss + k];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o, 64);
      if (lane == 0) rs[m] = e.ss_in ? 1.0f / sqrtf(t * (1.0f / (float)K) + e.eps) : 1.f;
    }
    __syncthreads();
  }
  auto sum4 = [&](int m, int n) {  // the S partials of 4 columns, added in split order
    float4 v = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < S; s0 += 4) {
      u32x4v q[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < S)
          q[j] = __builtin_amdgcn_raw_buffer_load_b128(pr, (uint32_t)((((size_t)(s0 + j) * M + m) * N + n) * 4), 0,
                                                       WIDE_SC1);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (s0 + j < S) {
          v.x += __uint_as_float(q[j][0]);
          v.y += __uint_as_float(q[j][1]);
          v.z += __uint_as_float(q[j][2]);
          v.w += __uint_as_float(q[j][3]);
        }
    }
    return v;
  };
  if constexpr (EPI == EPI_SWIGLU) {
    // packed rows 32i + j (gate, j < 16) and 32i + 16 + j (up) give output column n0/2 + 16i + j
    for (int x = tid; x < M * 16; x += blockDim.x) {
      const int m = x >> 4, q = x & 15, i = q >> 2, j4 = (q & 3) * 4;
      const float4 gt = sum4(m, n0 + 32 * i + j4), up = sum4(m, n0 + 32 * i + 16 + j4);
      const float sc = rs[m];
      const size_t o = (size_t)m * e.ldo + (n0 >> 1) + 16 * i + j4;
      split16(silu(gt.x * sc) * (up.x * sc), (f16*)e.out, (f16*)e.olo, o);
      split16(silu(gt.y * sc) * (up.y * sc), (f16*)e.out, (f16*)e.olo, o + 1);
      split16(silu(gt.z * sc) * (up.z * sc), (f16*)e.out, (f16*)e.olo, o + 2);
      split16(silu(gt.w * sc) * (up.w * sc), (f16*)e.out, (f16*)e.olo, o + 3);
    }
  } else {
    // 32 threads (half a wave) per row, 4 columns each
    for (int x = tid; x < ((M + 15) & ~15) * 32; x += blockDim.x) {
      const int m = x >> 5, n = n0 + 4 * (x & 31);
      const bool in = m < M;  // uniform over each half wave
      float4 v = {0.f, 0.f, 0.f, 0.f};
      if (in) v = sum4(m, n);
      if constexpr (EPI == EPI_STORE) {
        if (in) {
          const float sc = rs[m];
          *(float4*)((float*)e.out + (size_t)m * e.ldo + n) = float4{v.x * sc, v.y * sc, v.z * sc, v.w * sc};
        }
      } else {
        float q = 0.f;
        if (in) {
          float4* hp = (float4*)(e.h + (size_t)m * N + n);
          float4 hv = *hp;
          hv.x += v.x; hv.y += v.y; hv.z += v.z; hv.w += v.w;
          *hp = hv;
          if (e.o16) {
            const size_t o = (size_t)m * N + n;
            split16(hv.x, (f16*)e.o16, (f16*)e.olo2, o);
            split16(hv.y, (f16*)e.o16, (f16*)e.olo2, o + 1);
            split16(hv.z, (f16*)e.o16, (f16*)e.olo2, o + 2);
            split16(hv.w, (f16*)e.o16, (f16*)e.olo2, o + 3);
          }
          q = (hv.x * hv.x + hv.y * hv.y) + (hv.z * hv.z + hv.w * hv.w);
        }
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
        if (in && e.ss_out && (x & 31) == 0) e.ss_out[(size_t)m * (N / 128) + (n0 >> 7)] = q;
      }
    }
  }
}

// The activation fragments of a K step are all requested before its first
// MFMA, so their LDS round trips overlap (one per MFMA otherwise); with 8 or
// more fragments a wave keeps two weight chunks in flight instead of three,
// which holds it at 120 VGPRs (four waves per SIMD).  On the 7B shapes at 64
// rows: gate|up 54.0 -> 50.8 us, QKV 32.7 -> 31.6 us, down 29.3 -> 25.5 us.
// The reduction fused into the last split (EPI_STORE / _SWIGLU / _RESID)
// measured 1-2 us faster per projection than GEMM + reduction kernel at 16
// rows and 1-5 us slower at 64, where the O and down projections' 32 tiles
// then reduce on 32 CUs; the engine uses it up to 16 rows.
template <int MB, int LO, int EPI>
__global__ __launch_bounds__(512) void k_gemm_wide(const f16* __restrict__ xhi, const f16* __restrict__ xlo,
                                                   const f16* __restrict__ W, int M, int K,
                                                   float* __restrict__ part, int N, WideEpi ep) {
  constexpr int NX = LO == 2 ? 2 : 1;               // activation arrays (hi, lo)
  constexpr int XCH = NX * MB * 16 * 16;             // 16-byte pieces of one staged chunk
  constexpr int XPT = (XCH + 511) / 512;             // pieces per thread
  constexpr int WP = MB * NX >= 6 ? 2 : WIDE_WP;     // weight chunks in flight
  extern __shared__ __attribute__((aligned(16))) f16 xs[];  // [2 stages][NX][MB*16][WIDE_LDK]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * WIDE_ROWS + wave * 16;
  const int nch = K >> 7, S = gridDim.y, sp = blockIdx.y;
  const int s0 = sp * nch / S, s1 = (sp + 1) * nch / S, n = s1 - s0;
  // the split's chunks in rotated order, by tile index / 8: the workgroups an XCD
  // runs at once (ids equal mod 8) start at different columns of their rows.
  // Measured on the 7B shapes: 1-5% faster at 16 rows (down 20.7 -> 19.6 us),
  // 0-1.5% at 64; rotating by the tile index itself was slower for gate|up.
  const int rot = n > 0 ? (int)((blockIdx.x >> 3) % (unsigned)n) : 0;
  auto chunk = [&](int t) { const int u = t + rot; return s0 + (u >= n ? u - n : u); };

  // W in fragment order: this wave's strip, lane's 16 bytes of each block
  const f16* wstrip = W + (size_t)(n0 / 16) * (K >> 7) * 2048 + lane * 8;
  uint4 wr[WP][4];
  // activation staging, up to 4 pieces of 16 bytes per thread (named registers:
  // an array here ends up on the stack).  Piece e = tid + 512 q: array
  // e / (MB*256), token row (e / 16) % (MB*16) (rows past M read row M-1: they
  // only feed token columns that are never stored), 16-byte column e % 16.
  static_assert(XPT <= 4, "at most 4 staging pieces per thread");
  uint4 x0 = {0u, 0u, 0u, 0u}, x1 = x0, x2 = x0, x3 = x0;
#define AMS_WIDE_XLOAD1(q, xq, c)                                                                  \
  do {                                                                                             \
    const int e_ = tid + 512 * (q);                                                                \
    if ((q) < XPT && (XCH % 512 == 0 || e_ < XCH)) {                                               \
      const int arr_ = e_ / (MB * 256), row_ = (e_ >> 4) % (MB * 16), col_ = e_ & 15;              \
      xq = *(const uint4*)((arr_ ? xlo : xhi) + (size_t)(row_ < M ? row_ : M - 1) * K + ((c) << 7) + col_ * 8); \
    }                                                                                              \
  } while (0)
#define AMS_WIDE_XSTORE1(q, xq, stage)                                                             \
  do {                                                                                             \
    const int e_ = tid + 512 * (q);                                                                \
    if ((q) < XPT && (XCH % 512 == 0 || e_ < XCH)) {                                               \
      const int arr_ = e_ / (MB * 256), row_ = (e_ >> 4) % (MB * 16), col_ = e_ & 15;              \
      *(uint4*)(xs + ((size_t)((stage) * NX + arr_) * MB * 16 + row_) * WIDE_LDK + col_ * 8) = xq; \
    }                                                                                              \
  } while (0)
#define AMS_WIDE_XLOAD(c) \
  do { AMS_WIDE_XLOAD1(0, x0, c); AMS_WIDE_XLOAD1(1, x1, c); AMS_WIDE_XLOAD1(2, x2, c); AMS_WIDE_XLOAD1(3, x3, c); } while (0)
#define AMS_WIDE_XSTORE(stage) \
  do { AMS_WIDE_XSTORE1(0, x0, stage); AMS_WIDE_XSTORE1(1, x1, stage); AMS_WIDE_XSTORE1(2, x2, stage); AMS_WIDE_XSTORE1(3, x3, stage); } while (0)

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // one K chunk t: its MFMAs from stage t & 1 and weights w, then staging chunk
  // t+1, the activation loads of chunk t+2 and the weight loads of chunk t+WP
  // (into w), each where that chunk exists.  The activation loads go out
  // before the weight loads: vmcnt retires in issue order, so staging chunk
  // t+2 next round waits only for loads older than the newest weight chunk.
  auto step = [&](int t, uint4 (&w)[4], bool st1, bool ld2, bool ldw) __attribute__((always_inline)) {
    const f16* xb = xs + (size_t)((t & 1) * NX) * MB * 16 * WIDE_LDK;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      half8 bf[NX][MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int a = 0; a < NX; ++a)
          bf[a][mb] = *(const half8*)(xb + (size_t)(a * MB * 16 + mb * 16 + r) * WIDE_LDK + 32 * i + 8 * g);
      const half8 wf = as_half8(w[i]);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int a = 0; a < NX; ++a)
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wf, bf[a][mb], acc[mb], 0, 0, 0);
    }
    if (st1) AMS_WIDE_XSTORE((t + 1) & 1);
    if (ld2) AMS_WIDE_XLOAD(chunk(t + 2));
    __builtin_amdgcn_sched_barrier(0);  // keep the issue order
    if (ldw) wide_wload_fo(w, wstrip, chunk(t + WP));
    __syncthreads();
  };
  int t = 0;
  if (n >= 2 * WP) {
    // Every chunk the prologue and the steps of this loop load exists, so
    // their loads are unconditional and issued in one order (a step's
    // activation loads, then its weight loads; the prologue X(c), W(c + WP - 2)
    // for c = 2 - WP .. 1): the loads in flight at the loop head are the same
    // from either edge, and the compiler's waits count them exactly instead of
    // draining them (with conditional loads each step waited for the weights
    // it had just requested).  Measured on the 7B decoder: 64-row decode 44.4
    // -> 44.0 ms per step, 16-row 56-token decode 223.0 -> 222.1 ms.
#pragma unroll
    for (int c = 2 - WP; c <= 1; ++c) {
      if (c >= 0) AMS_WIDE_XLOAD(chunk(c));
      __builtin_amdgcn_sched_barrier(0);
      wide_wload_fo(wr[c + WP - 2], wstrip, chunk(c + WP - 2));
      __builtin_amdgcn_sched_barrier(0);
      if (c == 0) AMS_WIDE_XSTORE(0);  // before the staging registers take chunk 1
    }
    __syncthreads();
    for (; t + 2 * WP <= n; t += WP) {
#pragma unroll
      for (int p = 0; p < WP; ++p) step(t + p, wr[p], true, true, true);
    }
  } else {
#pragma unroll
    for (int p = 0; p < WP; ++p)
      if (p < n) wide_wload_fo(wr[p], wstrip, chunk(p));
    AMS_WIDE_XLOAD(chunk(0));
    AMS_WIDE_XSTORE(0);
    if (n > 1) AMS_WIDE_XLOAD(chunk(1));
    __syncthreads();
  }
  // the remaining steps (fewer than 2 WP with the loop above)
  for (; t < n; t += WP) {
#pragma unroll
    for (int p = 0; p < WP; ++p)
      if (t + p < n) step(t + p, wr[p], t + p + 1 < n, t + p + 2 < n, t + p + WP < n);
  }

#undef AMS_WIDE_XLOAD1
#undef AMS_WIDE_XSTORE1
#undef AMS_WIDE_XLOAD
#undef AMS_WIDE_XSTORE

  // lane (r, g) holds rows n0 + 4g + i for token mb*16 + r
  if constexpr (EPI == EPI_PART) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int tok = mb * 16 + r;
      if (tok >= M) continue;
      float* dst = part + ((size_t)sp * M + tok) * N + n0 + 4 * g;
      *(float4*)dst = float4{acc[mb][0], acc[mb][1], acc[mb][2], acc[mb][3]};
    }
  } else {
    __shared__ int last;
    const __amdgpu_buffer_rsrc_t pr = wide_rsrc(part, (uint32_t)((size_t)S * M * N * 4));
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int tok = mb * 16 + r;
      if (tok >= M) continue;
      __builtin_amdgcn_raw_buffer_store_b128(u32x4v{__float_as_uint(acc[mb][0]), __float_as_uint(acc[mb][1]),
                                                    __float_as_uint(acc[mb][2]), __float_as_uint(acc[mb][3])},
                                             pr, (uint32_t)((((size_t)sp * M + tok) * N + n0 + 4 * g) * 4), 0,
                                             WIDE_SC1);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's partial sums are stored
    __syncthreads();
    if (tid == 0) {
      unsigned* c = ep.cnt + blockIdx.x;
      const bool l = __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(S - 1);
      if (l) __hip_atomic_store(c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // every split is in
      last = l;
    }
    __syncthreads();
    if (last) wide_reduce<EPI>(ep, pr, S, M, N, K, blockIdx.x * WIDE_ROWS);
  }
}

template <int MB, int LO, int EPI>
static hipError_t launch_wide(const f16* x, const f16* xlo, const f16* W, int M, int N, int K, int splits,
                              float* part, const WideEpi& ep, hipStream_t s) {
  const size_t lds = (size_t)2 * (LO == 2 ? 2 : 1) * MB * 16 * WIDE_LDK * sizeof(f16);
  hipLaunchKernelGGL((k_gemm_wide<MB, LO, EPI>), dim3(N / WIDE_ROWS, splits), dim3(512), lds, s, x, xlo, W, M, K,
                     part, N, ep);
  return hipGetLastError();
}

template <int EPI>
static hipError_t wide_epi(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                           const WideEpi& ep, hipStream_t s) {
  const f16 *x = (const f16*)u, *xl = (const f16*)ulo, *w = (const f16*)W;
  if (!ulo) {
    if (M <= 16) return launch_wide<1, 0, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
    if (M <= 32) return launch_wide<2, 0, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
    if (M <= 48) return launch_wide<3, 0, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
    return launch_wide<4, 0, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
  }
  if (M <= 16) return launch_wide<1, 2, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
  if (M <= 32) return launch_wide<2, 2, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
  if (M <= 48) return launch_wide<3, 2, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
  return launch_wide<4, 2, EPI>(x, xl, w, M, N, K, splits, part, ep, s);
}

static bool wide_shape_ok(int M, int N, int K, int splits) {
  return M <= 64 && N % WIDE_ROWS == 0 && K % 128 == 0 && splits >= 1 && (K >> 7) >= splits;
}

hipError_t gemm_wide(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                     hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!wide_shape_ok(M, N, K, splits)) return hipErrorInvalidValue;
  return wide_epi<EPI_PART>(u, ulo, W, M, N, K, splits, part, WideEpi{}, s);
}

hipError_t gemm_wide_reduce(int epi, const void* u, const void* ulo, const void* W, int M, int N, int K, int splits,
                            float* part, unsigned* counters, void* out, void* olo, int ldo, float* h, void* o16,
                            void* olo2, float* ss_out, const float* ss_in, float eps, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!wide_shape_ok(M, N, K, splits) || !counters || !part) return hipErrorInvalidValue;
  if ((size_t)splits * M * N * 4 >= (size_t)1 << 31) return hipErrorInvalidValue;  // 32-bit buffer offsets
  WideEpi ep{counters, out, olo, ldo, h, o16, olo2, ss_out, ss_in, eps};
  switch (epi) {
    case EPI_STORE:
      if (!out || ldo < N) return hipErrorInvalidValue;
      return wide_epi<EPI_STORE>(u, ulo, W, M, N, K, splits, part, ep, s);
    case EPI_SWIGLU:
      if (!out || N % (2 * GU_BLOCK) != 0 || ldo < N / 2) return hipErrorInvalidValue;
      return wide_epi<EPI_SWIGLU>(u, ulo, W, M, N, K, splits, part, ep, s);
    case EPI_RESID:
      if (!h || (olo2 && !o16)) return hipErrorInvalidValue;
      return wide_epi<EPI_RESID>(u, ulo, W, M, N, K, splits, part, ep, s);
    default:
      return hipErrorInvalidValue;
  }
}

// 1/rms of row m from the partial sums of squares k_part_resid left for it
// (ss[m][0..nss), added in a fixed order), shared with the whole block;
// 1 when ss is NULL.  Every thread of the block calls it.
__device__ float row_rstd(const float* __restrict__ ss, int nss, int m, float inv_n, float eps) {
  __shared__ float r;
  if (!ss) return 1.f;
  if (threadIdx.x < 64) {
    float t = 0.f;
    for (int k = threadIdx.x; k < nss; k += 64) t += ss[(size_t)m * nss + k];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o, 64);
    if (threadIdx.x == 0) r = 1.0f / sqrtf(t * inv_n + eps);
  }
  __syncthreads();
  return r;
}

// out[m][n] = sum_s part[s][m][n] (splits added in order), times the row's
// 1/rms when ss is given (N a multiple of 256: a block lies in one row)
__global__ __launch_bounds__(256) void k_part_store(const float* __restrict__ part, int splits, size_t MN, int N,
                                                    const float* __restrict__ ss, int nss, float inv_n, float eps,
                                                    float* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  float v = 0.f;
  if (i < MN)
    for (int sp = 0; sp < splits; ++sp) v += part[sp * MN + i];
  // the row's scale after the partial loads are issued: both arrive in one round trip
  const float sc = row_rstd(ss, nss, (int)((size_t)blockIdx.x * blockDim.x / N), inv_n, eps);
  if (i < MN) out[i] = v * sc;
}

// a[m][c] = silu(gate) * up for the packed gate/up rows of output column c
// (16-row interleave), as an fp16 pair (out, olo); gate and up times the row's
// 1/rms when ss is given (N/2 a multiple of 256)
__global__ __launch_bounds__(256) void k_part_swiglu(const float* __restrict__ part, int splits, int M, int N,
                                                     const float* __restrict__ ss, int nss, float inv_n, float eps,
                                                     f16* __restrict__ out, f16* __restrict__ olo) {
  const int F = N / 2;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool in = i < (size_t)M * F;
  float gt = 0.f, up = 0.f;
  if (in) {
    const int m = (int)(i / F), c = (int)(i % F);
    const size_t gi = (size_t)m * N + (size_t)(c / GU_BLOCK) * 2 * GU_BLOCK + c % GU_BLOCK, MN = (size_t)M * N;
    for (int sp = 0; sp < splits; ++sp) {
      gt += part[sp * MN + gi];
      up += part[sp * MN + gi + GU_BLOCK];
    }
  }
  // the row's scale after the partial loads are issued: both arrive in one round trip
  const float sc = row_rstd(ss, nss, (int)((size_t)blockIdx.x * blockDim.x / F), inv_n, eps);
  if (in) split16(silu(gt * sc) * (up * sc), out, olo, i);
}

hipError_t part_store(const float* part, int splits, int M, int N, float* out, hipStream_t s, const float* ss,
                      int d, float eps) {
  if (M <= 0) return hipSuccess;
  if (ss && (N % 256 != 0 || d <= 0 || d % 256 != 0)) return hipErrorInvalidValue;
  const size_t MN = (size_t)M * N;
  hipLaunchKernelGGL(k_part_store, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, part, splits, MN, N, ss,
                     d / 128, ss ? 1.0f / (float)d : 0.f, eps, out);
  return hipGetLastError();
}

hipError_t part_swiglu(const float* part, int splits, int M, int N, void* out, void* olo, hipStream_t s,
                       const float* ss, int d, float eps) {
  if (M <= 0) return hipSuccess;
  if (N % (2 * GU_BLOCK) != 0) return hipErrorInvalidValue;
  if (ss && ((N / 2) % 256 != 0 || d <= 0 || d % 256 != 0)) return hipErrorInvalidValue;
  const size_t MF = (size_t)M * (N / 2);
  hipLaunchKernelGGL(k_part_swiglu, dim3((unsigned)((MF + 255) / 256)), dim3(256), 0, s, part, splits, M, N, ss,
                     d / 128, ss ? 1.0f / (float)d : 0.f, eps, (f16*)out, (f16*)olo);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// split-K decode GEMV: partial sums of `splits` K ranges, then a reduction

hipError_t gemm_part(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                     hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (M > 64 || splits < 1 || (K >> 7) < splits) return hipErrorInvalidValue;
  const SkinnyArgs a{(const f16*)u, (const f16*)ulo, 0.f, (const f16*)W, M, K, part, N, nullptr, nullptr};
  if (!ulo) {
    if (M <= 16) return launch_skinny<1, 1, EPI_PART, false, 0>(a, N, s, splits);
    if (M <= 32) return launch_skinny<1, 2, EPI_PART, false, 0>(a, N, s, splits);
    if (M <= 48) return launch_skinny<1, 3, EPI_PART, false, 0>(a, N, s, splits);
    return launch_skinny<1, 4, EPI_PART, false, 0>(a, N, s, splits);
  }
  if (M <= 8) return launch_skinny<1, 1, EPI_PART, false, 1>(a, N, s, splits);
  if (M <= 16) return launch_skinny<1, 1, EPI_PART, false, 2>(a, N, s, splits);
  if (M <= 32) return launch_skinny<1, 2, EPI_PART, false, 2>(a, N, s, splits);
  if (M <= 48) return launch_skinny<1, 3, EPI_PART, false, 2>(a, N, s, splits);
  return launch_skinny<1, 4, EPI_PART, false, 2>(a, N, s, splits);
}

// h[m][n] += sum_s part[s][m][n] (splits in order), and the fp16 pair of the
// updated row when o16 is non-NULL; with ss, each block (256 columns of one
// row: N a multiple of 256) also leaves the sums of squares of its new values
// per 128 columns at ss[2 blockIdx ..], i.e. ss[m][n / 128], for the next
// projection's RMSNorm
__global__ __launch_bounds__(256) void k_part_resid(const float* __restrict__ part, int splits, int M, int N,
                                                    float* __restrict__ h, f16* __restrict__ o16,
                                                    f16* __restrict__ olo, float* __restrict__ ss) {
  __shared__ float wsq[4];
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t MN = (size_t)M * N;
  float hn = 0.f;
  if (i < MN) {
    float v = 0.f;
    for (int sp = 0; sp < splits; ++sp) v += part[sp * MN + i];
    hn = h[i] + v;
    h[i] = hn;
    if (o16) split16(hn, o16, olo, i);
  }
  if (!ss) return;
  float q = hn * hn;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  if ((threadIdx.x & 63) == 0) wsq[threadIdx.x >> 6] = q;
  __syncthreads();
  if (threadIdx.x < 2) ss[2 * blockIdx.x + threadIdx.x] = wsq[2 * threadIdx.x] + wsq[2 * threadIdx.x + 1];
}

hipError_t part_resid(const float* part, int splits, int M, int N, float* h, void* o16, void* olo, hipStream_t s,
                      float* ss) {
  if (M <= 0) return hipSuccess;
  if ((olo && !o16) || (ss && N % 256 != 0)) return hipErrorInvalidValue;
  const size_t MN = (size_t)M * N;
  hipLaunchKernelGGL(k_part_resid, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, part, splits, M, N, h,
                     (f16*)o16, (f16*)olo, ss);
  return hipGetLastError();
}

template <int EPI>
static hipError_t gemm_epi(int ct, const void* u, const void* W, int M, int N, int K, void* out, int ldo,
                           hipStream_t s, const void* ulo, void* o16, void* olo) {
  const bool pair = ulo || o16 || olo;
  if (pair) {  // the fp16-pair forms belong to the decode GEMV only
    if (ct != DT_F16 || M > 64) return hipErrorInvalidValue;
    if (o16 && EPI != EPI_RESID) return hipErrorInvalidValue;
    if (olo && EPI == EPI_STORE) return hipErrorInvalidValue;
    if (olo && EPI == EPI_RESID && !o16) return hipErrorInvalidValue;
  }
  if (ct == DT_F32) {
    hipLaunchKernelGGL((k_gemm_f32<EPI>), dim3(N / FBN, (M + FBM - 1) / FBM), dim3(256), 0, s,
                       (const float*)u, (const float*)W, M, K, out, ldo);
    return hipGetLastError();
  }
  if (M <= 64) {
    const SkinnyArgs a{(const f16*)u, (const f16*)ulo, 0.f, (const f16*)W, M, K, out, ldo, (f16*)o16, (f16*)olo};
    return skinny_dispatch<EPI, false>(a, N, s);
  }
  // 256 x 256 tiles from 160 of them on (five in eight CUs busy), 128 x 128 below: on the 7B
  // shapes the big tiles won at 172 (gate|up, 288 tokens) and 192 (QKV, 1024 tokens) tiles and
  // lost at 96 and 64
  if (N % GBN == 0 && (size_t)(N / GBN) * ((M + GBM - 1) / GBM) >= 160) {
    if constexpr (EPI == EPI_STORE)
      if (big_narrow(M, N)) return launch_big<EPI, 192>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
    const int nb = big_main_cols(M, N) * GBN;
    hipError_t e = launch_big<EPI>((const f16*)u, (const f16*)W, M, nb, K, out, ldo, s);
    if (e != hipSuccess || nb == N) return e;
    // the weight rows past nb in 256 x 128 tiles (output columns nb / 2 on for SwiGLU):
    // the 7B gate|up remainder at 1,024 tokens took 81.9 us as 128 x 128 tiles
    void* o2 = EPI == EPI_SWIGLU ? (void*)((f16*)out + nb / 2) : (void*)((float*)out + nb);
    return launch_big<EPI, 128>((const f16*)u, (const f16*)W + (size_t)nb * K, M, N - nb, K, o2, ldo, s);
  }
  hipLaunchKernelGGL((k_gemm_tiled<EPI>), dim3(N / TBN, (M + TBM - 1) / TBM), dim3(256), 0, s,
                     (const f16*)u, (const f16*)W, M, K, out, ldo);
  return hipGetLastError();
}

bool gemm_qkv_fusable(int M, int N, int dh, int d) {
  if (M <= 64 || (dh != 64 && dh != 128) || d % 256 != 0 || N != 3 * d) return false;
  if ((size_t)(N / GBN) * ((M + GBM - 1) / GBM) < 160) return false;  // gemm() takes the tiled kernel
  return !big_narrow(M, N) && big_main_cols(M, N) == N / GBN;       // ... or other tile widths
}

hipError_t gemm_qkv_kv(const void* u, const void* W, int M, int K, float* qkv, const KvEpi& kv, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if ((kv.dh != 64 && kv.dh != 128) || kv.d <= 0 || kv.d % 256 != 0 || K % GBK != 0 || !kv.tok_base || !kv.tok_pos ||
      !kv.k || !kv.v || !kv.rope)
    return hipErrorInvalidValue;
  return launch_big<EPI_QKV>((const f16*)u, (const f16*)W, M, 3 * kv.d, K, qkv, 3 * kv.d, s, 1, kv);
}

hipError_t gemm_big_part(const void* u, const void* W, int M, int N, int K, int splits, float* part, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (N % GBN != 0 || K % GBK != 0 || splits < 1 || splits > K / GBK) return hipErrorInvalidValue;
  return launch_big<EPI_PART>((const f16*)u, (const f16*)W, M, N, K, part, N, s, splits);
}

hipError_t gemm_big(int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo, hipStream_t s,
                    int bn) {
  if (M <= 0) return hipSuccess;
  if (bn == 192) {
    if (epi != EPI_STORE || N % 192 != 0 || K % GBK != 0) return hipErrorInvalidValue;
    return launch_big<EPI_STORE, 192>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
  }
  if (bn == 128) {
    if (N % 128 != 0 || K % GBK != 0) return hipErrorInvalidValue;
    switch (epi) {
      case EPI_STORE: return launch_big<EPI_STORE, 128>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
      case EPI_RESID: return launch_big<EPI_RESID, 128>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
      default: return launch_big<EPI_SWIGLU, 128>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
    }
  }
  if (bn != GBN || N % GBN != 0 || K % GBK != 0) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE: return launch_big<EPI_STORE>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
    case EPI_RESID: return launch_big<EPI_RESID>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
    default: return launch_big<EPI_SWIGLU>((const f16*)u, (const f16*)W, M, N, K, out, ldo, s);
  }
}

hipError_t gemm(int ct, int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo,
                hipStream_t s, const void* ulo, void* o16, void* olo) {
  if (M <= 0) return hipSuccess;
  switch (epi) {
    case EPI_STORE: return gemm_epi<EPI_STORE>(ct, u, W, M, N, K, out, ldo, s, ulo, o16, olo);
    case EPI_RESID: return gemm_epi<EPI_RESID>(ct, u, W, M, N, K, out, ldo, s, ulo, o16, olo);
    default: return gemm_epi<EPI_SWIGLU>(ct, u, W, M, N, K, out, ldo, s, ulo, o16, olo);
  }
}

hipError_t gemv_rmsnorm(int ct, int epi, const void* hhi, float eps, const void* W, int M, int N, int K, void* out,
                        int ldo, hipStream_t s, const void* hlo, void* o16, void* olo) {
  if (M <= 0) return hipSuccess;
  if (ct != DT_F16 || M > 16) return hipErrorInvalidValue;
  if (o16 && epi != EPI_RESID) return hipErrorInvalidValue;
  if (olo && (epi == EPI_STORE || (epi == EPI_RESID && !o16))) return hipErrorInvalidValue;
  const SkinnyArgs a{(const f16*)hhi, (const f16*)hlo, eps, (const f16*)W, M, K, out, ldo, (f16*)o16, (f16*)olo};
  switch (epi) {
    case EPI_STORE: return skinny_dispatch<EPI_STORE, true>(a, N, s);
    case EPI_RESID: return skinny_dispatch<EPI_RESID, true>(a, N, s);
    default: return skinny_dispatch<EPI_SWIGLU, true>(a, N, s);
  }
}

}  // namespace ams

// Attention over the cached context.
//
// K/V slab of one layer: K and V each [row][head][capacity][head_dim] in the
// model dtype, so the keys of one (row, head) are one contiguous stream.
//
//  * k_kv_append:     new tokens of a pass -> rotate k (RoPE), write k and v
//                     at their absolute positions.
//  * k_attn_prefill_mfma (fp16) / k_attn_prefill (fp32): causal attention of
//                     a pass's tokens (a row's new segment at positions
//                     pos..pos+n-1) over keys 0..pos+n-1 of that row, K/V
//                     tiles staged in LDS, online softmax; the fp16 kernel
//                     runs both products on MFMA.
//  * k_attn_decode:   one query per row at position p = lens[b] + jpos (a
//                     fed-back action token).  Appends its own K/V, then
//                     each workgroup covers one split of the keys: lane-per-key
//                     scores, wavefront-shuffle online softmax, and a P.V
//                     pass with lanes over (key subgroup, 8-dim chunk).  The
//                     split partials (m, l, acc) are merged by k_attn_merge
//                     with log-sum-exp weights.
#include "common.h"
#include "kernels.h"

namespace ams {

__device__ __forceinline__ int find_seg(const int32_t* off, int n_seg, int i) {
  int lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// 8 consecutive elements as floats
__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load8(const f16* p, float* v) {
  const half8 a = __builtin_bit_cast(half8, *(const uint4*)p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
}

// ----------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void k_kv_append(const float* __restrict__ qkv, const int32_t* __restrict__ row,
                                                   const int32_t* __restrict__ pos, const int32_t* __restrict__ off,
                                                   int n_seg, int H, int dh, int cap, const float2* __restrict__ rope,
                                                   T* __restrict__ kslab, T* __restrict__ vslab) {
  const int i = blockIdx.x;
  const int s = find_seg(off, n_seg, i);
  const int b = row[s], p = pos[s] + (i - off[s]);
  const int d = H * dh, half = dh / 2;
  const float* k = qkv + (size_t)i * 3 * d + d;
  const float* v = k + d;
  for (int e = threadIdx.x; e < H * half; e += blockDim.x) {
    const int h = e / half, ii = e % half;
    const float2 cs = rope[(size_t)p * half + ii];
    const float a = k[h * dh + ii], c = k[h * dh + ii + half];
    T* dst = kslab + (((size_t)b * H + h) * cap + p) * dh;
    st<T>(dst, ii, a * cs.x - c * cs.y);
    st<T>(dst, ii + half, a * cs.y + c * cs.x);
  }
  for (int e = threadIdx.x; e < d; e += blockDim.x) {
    const int h = e / dh, dd = e % dh;
    st<T>(vslab + (((size_t)b * H + h) * cap + p) * dh, dd, v[e]);
  }
}

hipError_t kv_append(int ct, const float* qkv, Segs sg, int H, int dh, int cap, const float2* rope,
                     void* kslab, void* vslab, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  if (ct == DT_F32)
    hipLaunchKernelGGL(k_kv_append<float>, dim3(sg.n_tok), dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off,
                       sg.n_seg, H, dh, cap, rope, (float*)kslab, (float*)vslab);
  else
    hipLaunchKernelGGL(k_kv_append<f16>, dim3(sg.n_tok), dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off,
                       sg.n_seg, H, dh, cap, rope, (f16*)kslab, (f16*)vslab);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------

template <typename T, int DH>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ qkv, const int32_t* __restrict__ row,
                                                      const int32_t* __restrict__ pos,
                                                      const int32_t* __restrict__ off, int H, int cap,
                                                      const float2* __restrict__ rope, const T* __restrict__ kslab,
                                                      const T* __restrict__ vslab, T* __restrict__ o, float scale) {
  constexpr int QT = 64, KT = 32, HALF = DH / 2, DPT = DH / 4;
  __shared__ float Qs[QT][DH + 1];
  __shared__ float Ks[KT][DH + 1];
  __shared__ float Vs[KT][DH];
  __shared__ float Ps[QT][KT + 1];
  const int s = blockIdx.z, h = blockIdx.y, tid = threadIdx.x;
  const int b = row[s], p0 = pos[s], t0 = off[s], n = off[s + 1] - off[s];
  const int q_lo = blockIdx.x * QT;
  if (q_lo >= n) return;  // uniform across the workgroup
  const int d = H * DH;

  for (int e = tid; e < QT * HALF; e += blockDim.x) {
    const int qi = e / HALF, ii = e % HALF;
    float x0 = 0.f, x1 = 0.f;
    if (q_lo + qi < n) {
      const int tok = t0 + q_lo + qi, p = p0 + q_lo + qi;
      const float* q = qkv + (size_t)tok * 3 * d + h * DH;
      const float2 cs = rope[(size_t)p * HALF + ii];
      const float a = q[ii], c = q[ii + HALF];
      x0 = (a * cs.x - c * cs.y) * scale;
      x1 = (a * cs.y + c * cs.x) * scale;
    }
    Qs[qi][ii] = x0;
    Qs[qi][ii + HALF] = x1;
  }

  const int qi = tid >> 2, sub = tid & 3;
  const bool valid = q_lo + qi < n;
  const int qpos = valid ? p0 + q_lo + qi : -1;
  const int kv_end = p0 + (n < q_lo + QT ? n : q_lo + QT);  // exclusive
  const T* Kb = kslab + ((size_t)b * H + h) * cap * DH;
  const T* Vb = vslab + ((size_t)b * H + h) * cap * DH;
  float m = -INFINITY, l = 0.f, acc[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) acc[i] = 0.f;

  for (int k0 = 0; k0 < kv_end; k0 += KT) {
    __syncthreads();  // Qs ready on the first pass; Ks/Vs/Ps free on later ones
    for (int e = tid; e < KT * DH; e += blockDim.x) {
      const int kk = e / DH, dd = e % DH;
      const bool ok = k0 + kk < kv_end;
      Ks[kk][dd] = ok ? ld<T>(Kb, (size_t)(k0 + kk) * DH + dd) : 0.f;
      Vs[kk][dd] = ok ? ld<T>(Vb, (size_t)(k0 + kk) * DH + dd) : 0.f;
    }
    __syncthreads();
    float sc[KT / 4];
    float mx = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < KT / 4; ++jj) {
      const int kk = sub + 4 * jj, kp = k0 + kk;
      float t = -INFINITY;
      if (kp <= qpos && kp < kv_end) {
        t = 0.f;
#pragma unroll 16
        for (int dd = 0; dd < DH; ++dd) t = fmaf(Qs[qi][dd], Ks[kk][dd], t);
      }
      sc[jj] = t;
      mx = fmaxf(mx, t);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
    const float m_new = fmaxf(m, mx);
    const float alpha = (m_new == -INFINITY) ? 1.f : __expf(m - m_new);
    float ps = 0.f;
#pragma unroll
    for (int jj = 0; jj < KT / 4; ++jj) {
      const float pv = (sc[jj] == -INFINITY) ? 0.f : __expf(sc[jj] - m_new);
      Ps[qi][sub + 4 * jj] = pv;
      ps += pv;
    }
    ps += __shfl_xor(ps, 1, 64);
    ps += __shfl_xor(ps, 2, 64);
    l = l * alpha + ps;
    m = m_new;
#pragma unroll
    for (int i = 0; i < DPT; ++i) acc[i] *= alpha;
    __syncthreads();
    for (int kk = 0; kk < KT; ++kk) {
      const float pk = Ps[qi][kk];
#pragma unroll
      for (int i = 0; i < DPT; ++i) acc[i] = fmaf(pk, Vs[kk][sub * DPT + i], acc[i]);
    }
  }
  if (valid) {
    const float inv = 1.0f / l;
    T* dst = o + (size_t)(t0 + q_lo + qi) * d + h * DH + sub * DPT;
#pragma unroll
    for (int i = 0; i < DPT; ++i) st<T>(dst, i, acc[i] * inv);
  }
}

// ----------------------------------------------------------------------------
// fp16 prefill attention on MFMA (flash-attention style).
//
// Workgroup: 64 queries of one segment and head, 4 waves x 16 queries.
// Per 64-key tile: K [key][dh] and V^T [dh][key] staged in LDS (fp16);
// S = Q K^T with v_mfma_f32_16x16x32_f16 (A = Q fragments held in registers,
// rotated and scaled at load; B = K rows), online softmax in fp32 over the
// 16-lane groups that share a query, P written to LDS and read back in the
// A-operand layout, O += P V with B = V^T rows.  MFMA layouts (16x16x32):
// A lane (r, g) = A[r][8g..8g+7], B lane (r, g) = B[8g..8g+7][r],
// C lane (r, g) = C[4g+i][r], with r = lane & 15, g = lane >> 4.

template <int DH>
__global__ __launch_bounds__(256) void k_attn_prefill_mfma(const float* __restrict__ qkv,
                                                           const int32_t* __restrict__ row,
                                                           const int32_t* __restrict__ pos,
                                                           const int32_t* __restrict__ off, int H, int cap,
                                                           const float2* __restrict__ rope,
                                                           const f16* __restrict__ kslab,
                                                           const f16* __restrict__ vslab, f16* __restrict__ o,
                                                           float scale) {
  constexpr int QT = 64, KT = 64, HALF = DH / 2, KPAD = DH + 8, VPAD = KT + 8, PPAD = KT + 8;
  constexpr int NQI = DH / 32;  // 32-wide dim blocks of a head (MFMA k-steps of S)
  constexpr int NDJ = DH / 16;  // 16-wide dim blocks of O
  __shared__ __attribute__((aligned(16))) f16 Ks[KT * KPAD];
  __shared__ __attribute__((aligned(16))) f16 VT[DH * VPAD];
  __shared__ __attribute__((aligned(16))) f16 Ps[4 * 16 * PPAD];
  const int sg = blockIdx.z, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int b = row[sg], p0 = pos[sg], t0 = off[sg], n = off[sg + 1] - off[sg];
  const int q_lo = blockIdx.x * QT;
  if (q_lo >= n) return;  // uniform across the workgroup
  const int d = H * DH;
  const int kv_end = p0 + (n < q_lo + QT ? n : q_lo + QT);  // exclusive

  // Q fragments: this lane's query row r of the wave, dims 32i + 8g + e
  half8 qf[NQI];
  {
    const int qi = q_lo + wave * 16 + r;
    const bool ok = qi < n;
    const float* q = qkv + (size_t)(t0 + (ok ? qi : 0)) * 3 * d + h * DH;
    const float2* rp = rope + (size_t)(p0 + (ok ? qi : 0)) * HALF;
#pragma unroll
    for (int i = 0; i < NQI / 2; ++i) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dd = 32 * i + 8 * g + e;  // < HALF; its partner is dd + HALF
        const float a = ok ? q[dd] : 0.f, c = ok ? q[dd + HALF] : 0.f;
        const float2 cs = rp[dd];
        qf[i][e] = (f16)((a * cs.x - c * cs.y) * scale);
        qf[i + NQI / 2][e] = (f16)((a * cs.y + c * cs.x) * scale);
      }
    }
  }
  // query positions of this lane's C rows (4g + i)
  int qp[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qi = q_lo + wave * 16 + 4 * g + i;
    qp[i] = qi < n ? p0 + qi : -1;
  }

  float m[4], l[4];
  f32x4 acc[NDJ];
#pragma unroll
  for (int i = 0; i < 4; ++i) { m[i] = -INFINITY; l[i] = 0.f; }
#pragma unroll
  for (int j = 0; j < NDJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const f16* Kb = kslab + ((size_t)b * H + h) * cap * DH;
  const f16* Vb = vslab + ((size_t)b * H + h) * cap * DH;
  f16* Pw = Ps + wave * 16 * PPAD;
  constexpr int CH = DH / 8;  // 16-byte chunks per key row

  for (int kt = 0; kt < kv_end; kt += KT) {
    __syncthreads();  // previous tile's Ks / VT / Ps reads are done
    for (int c = tid; c < KT * CH; c += 256) {
      const int kk = c / CH, ch = c % CH;
      const bool ok = kt + kk < kv_end;
      uint4 kv = ok ? *(const uint4*)(Kb + (size_t)(kt + kk) * DH + ch * 8) : uint4{0u, 0u, 0u, 0u};
      uint4 vv = ok ? *(const uint4*)(Vb + (size_t)(kt + kk) * DH + ch * 8) : uint4{0u, 0u, 0u, 0u};
      *(uint4*)(Ks + kk * KPAD + ch * 8) = kv;
      const half8 vh = __builtin_bit_cast(half8, vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) VT[(ch * 8 + e) * VPAD + kk] = vh[e];
    }
    __syncthreads();

    // S for 4 blocks of 16 keys
    f32x4 sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      sc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < NQI; ++i) {
        const half8 kf = *(const half8*)(Ks + (kb * 16 + r) * KPAD + 32 * i + 8 * g);
        sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qf[i], kf, sc[kb], 0, 0, 0);
      }
    }
    // mask, online softmax per query row 4g+i (its 64 keys sit in the 16 lanes sharing g)
    float mx[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int key = kt + kb * 16 + r;
        if (key > qp[i] || key >= kv_end) sc[kb][i] = -INFINITY;
        v = fmaxf(v, sc[kb][i]);
      }
#pragma unroll
      for (int o_ = 1; o_ < 16; o_ <<= 1) v = fmaxf(v, __shfl_xor(v, o_, 64));
      mx[i] = v;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float m_new = fmaxf(m[i], mx[i]);
      const float alpha = (m_new == -INFINITY) ? 1.f : __expf(m[i] - m_new);
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const float pv = (sc[kb][i] == -INFINITY) ? 0.f : __expf(sc[kb][i] - m_new);
        sc[kb][i] = pv;
        rs += pv;
      }
#pragma unroll
      for (int o_ = 1; o_ < 16; o_ <<= 1) rs += __shfl_xor(rs, o_, 64);
      l[i] = l[i] * alpha + rs;
      m[i] = m_new;
#pragma unroll
      for (int j = 0; j < NDJ; ++j) acc[j][i] *= alpha;
    }
    // P (C layout) -> LDS [q][key] -> A layout
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) Pw[(4 * g + i) * PPAD + kb * 16 + r] = (f16)sc[kb][i];
    __syncthreads();
#pragma unroll
    for (int s2 = 0; s2 < KT / 32; ++s2) {
      const half8 pf = *(const half8*)(Pw + r * PPAD + 32 * s2 + 8 * g);
#pragma unroll
      for (int j = 0; j < NDJ; ++j) {
        const half8 vf = *(const half8*)(VT + (16 * j + r) * VPAD + 32 * s2 + 8 * g);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf, vf, acc[j], 0, 0, 0);
      }
    }
  }
  // O / l -> o[token][h*DH + dh]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qi = q_lo + wave * 16 + 4 * g + i;
    if (qi >= n) continue;
    const float inv = 1.0f / l[i];
    f16* dst = o + (size_t)(t0 + qi) * d + h * DH;
#pragma unroll
    for (int j = 0; j < NDJ; ++j) st<f16>(dst, 16 * j + r, acc[j][i] * inv);
  }
}

template <typename T>
static hipError_t prefill_t(const float* qkv, Segs sg, int H, int dh, int cap, const float2* rope, const void* k,
                            const void* v, void* o, hipStream_t s) {
  const dim3 grid((sg.max_len + 63) / 64, H, sg.n_seg);
  const float scale = 1.0f / sqrtf((float)dh);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_prefill<T, 64>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, cap, rope,
                       (const T*)k, (const T*)v, (T*)o, scale);
  else
    hipLaunchKernelGGL((k_attn_prefill<T, 128>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, cap, rope,
                       (const T*)k, (const T*)v, (T*)o, scale);
  return hipGetLastError();
}

hipError_t attn_prefill(int ct, const float* qkv, Segs sg, int H, int dh, int cap, const float2* rope,
                        const void* kslab, const void* vslab, void* o, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  if (ct == DT_F32) return prefill_t<float>(qkv, sg, H, dh, cap, rope, kslab, vslab, o, s);
  const dim3 grid((sg.max_len + 63) / 64, H, sg.n_seg);
  const float scale = 1.0f / sqrtf((float)dh);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_prefill_mfma<64>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, cap, rope,
                       (const f16*)kslab, (const f16*)vslab, (f16*)o, scale);
  else
    hipLaunchKernelGGL((k_attn_prefill_mfma<128>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, cap, rope,
                       (const f16*)kslab, (const f16*)vslab, (f16*)o, scale);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------

template <typename T> struct Raw;  // 16-byte chunks of T -> floats
template <> struct Raw<f16> {
  static constexpr int E = 8;
  static __device__ __forceinline__ void cvt(const uint4& r, float* v) {
    const half8 a = __builtin_bit_cast(half8, r);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
  }
};
template <> struct Raw<float> {
  static constexpr int E = 4;
  static __device__ __forceinline__ void cvt(const uint4& r, float* v) {
    v[0] = __uint_as_float(r.x); v[1] = __uint_as_float(r.y); v[2] = __uint_as_float(r.z); v[3] = __uint_as_float(r.w);
  }
};

// Waves per decode workgroup: 8 for 64-wide heads (one round covers 512
// positions), 4 for 128-wide heads (their K/V fragments need twice the registers).
template <int DH> constexpr int decode_waves() { return DH == 64 ? 8 : 4; }

template <typename T, int DH>
__global__ __launch_bounds__(64 * decode_waves<DH>()) void k_attn_decode(const float* __restrict__ qkv, const int32_t* __restrict__ lens,
                                                     int jpos, int H, int cap, int splits,
                                                     const float2* __restrict__ rope, T* __restrict__ kslab,
                                                     T* __restrict__ vslab, float* __restrict__ part,
                                                     T* __restrict__ o, float scale) {
  constexpr int HALF = DH / 2, NC = DH / 8, KS = 64 / NC;  // dim chunks of 8; key subgroups per wave
  constexpr int E = Raw<T>::E, KR = DH / E, VI = 64 / KS, VR = 8 / E;
  constexpr int NWV = decode_waves<DH>();
  __shared__ float qs[DH], kn[DH], vn[DH];
  __shared__ float wm[NWV], wl[NWV], wacc[NWV][DH];
  const int sp = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = H * DH;
  const int p = lens[b] + jpos;  // position of this pass's token
  const int T_ = p + 1;          // keys 0..p
  const int chunk = (cap + splits - 1) / splits;
  const int k0 = sp * chunk;
  const int k1 = (k0 + chunk < T_) ? k0 + chunk : T_;
  const float* qrow = qkv + (size_t)b * 3 * d + h * DH;

  const size_t bh = ((size_t)b * H + h) * cap;
  const T* Kb = kslab + bh * DH;
  const T* Vb = vslab + bh * DH;
  const int ks = lane / NC, dc = lane % NC;
  uint4 kraw[KR];
  uint4 vraw[VI][VR];
  // one block's K row (lane = key) and V chunks (lane = key subgroup x dim chunk)
  auto load_block = [&](int kb) {
    const int key = kb + lane;
    if (key < k1 && key != p) {
      const uint4* kr = (const uint4*)(Kb + (size_t)key * DH);
#pragma unroll
      for (int i = 0; i < KR; ++i) kraw[i] = kr[i];
    }
#pragma unroll
    for (int it = 0; it < VI; ++it) {
      const int kk = kb + it * KS + ks;
      if (kk < k1 && kk != p) {
        const uint4* vr = (const uint4*)(Vb + (size_t)kk * DH + dc * 8);
#pragma unroll
        for (int r = 0; r < VR; ++r) vraw[it][r] = vr[r];
      }
    }
  };
  // the first block's loads go out before the prologue, overlapping it
  const int kb0 = k0 + wave * 64;
  if (kb0 < k1) load_block(kb0);

  if (tid < HALF) {
    const float2 cs = rope[(size_t)p * HALF + tid];
    float a = qrow[tid], c = qrow[tid + HALF];
    qs[tid] = (a * cs.x - c * cs.y) * scale;
    qs[tid + HALF] = (a * cs.y + c * cs.x) * scale;
    a = qrow[d + tid];
    c = qrow[d + tid + HALF];
    // the stored (rounded) key is the one every later step reads; use it here too
    T r0, r1;
    st<T>(&r0, 0, a * cs.x - c * cs.y);
    st<T>(&r1, 0, a * cs.y + c * cs.x);
    kn[tid] = ld<T>(&r0, 0);
    kn[tid + HALF] = ld<T>(&r1, 0);
  }
  if (tid < DH) {
    T r;
    st<T>(&r, 0, qrow[2 * d + tid]);
    vn[tid] = ld<T>(&r, 0);
  }
  __syncthreads();
  if (k0 <= p && p < k1 && tid < DH) {
    st<T>(kslab + (bh + p) * DH, tid, kn[tid]);
    st<T>(vslab + (bh + p) * DH, tid, vn[tid]);
  }

  float m = -INFINITY, l = 0.f, acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;

  for (int kb = kb0; kb < k1; kb += NWV * 64) {
    if (kb != kb0) load_block(kb);
    const int key = kb + lane;
    float sc = -INFINITY;
    if (key < k1) {
      sc = 0.f;
      if (key == p) {
#pragma unroll 8
        for (int dd = 0; dd < DH; ++dd) sc = fmaf(qs[dd], kn[dd], sc);
      } else {
#pragma unroll
        for (int i = 0; i < KR; ++i) {
          float kv[E];
          Raw<T>::cvt(kraw[i], kv);
#pragma unroll
          for (int e = 0; e < E; ++e) sc = fmaf(qs[i * E + e], kv[e], sc);
        }
      }
    }
    const float m_new = fmaxf(m, wave_max(sc));
    const float alpha = __expf(m - m_new);  // m = -inf on the first block gives 0
    const float pl = (key < k1) ? __expf(sc - m_new) : 0.f;
    l = l * alpha + wave_sum(pl);
    m = m_new;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] *= alpha;
#pragma unroll
    for (int it = 0; it < VI; ++it) {
      const int kl = it * KS + ks;
      const float pk = __shfl(pl, kl, 64);
      const int kk = kb + kl;
      if (kk < k1) {
        float vv[8];
        if (kk == p) {
#pragma unroll
          for (int e = 0; e < 8; ++e) vv[e] = vn[dc * 8 + e];
        } else {
#pragma unroll
          for (int r = 0; r < VR; ++r) Raw<T>::cvt(vraw[it][r], vv + r * E);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(pk, vv[e], acc[e]);
      }
    }
  }
  // sum the key subgroups: lanes that share a dim chunk differ in the high bits
#pragma unroll
  for (int off_ = NC; off_ < 64; off_ <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], off_, 64);
  if (lane == 0) {
    wm[wave] = m;
    wl[wave] = l;
  }
  if (lane < NC)
#pragma unroll
    for (int e = 0; e < 8; ++e) wacc[wave][lane * 8 + e] = acc[e];
  __syncthreads();
  if (tid < DH) {
    float M = wm[0];
#pragma unroll
    for (int w = 1; w < NWV; ++w) M = fmaxf(M, wm[w]);
    float L = 0.f, Acc = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NWV; ++w) {
        const float f = __expf(wm[w] - M);
        L += wl[w] * f;
        Acc += wacc[w][tid] * f;
      }
    }
    if (splits == 1) {
      st<T>(o, (size_t)b * d + h * DH + tid, Acc / L);
    } else {
      float* out = part + (((size_t)b * H + h) * splits + sp) * (DH + 2);
      out[2 + tid] = Acc;
      if (tid == 0) {
        out[0] = M;
        out[1] = L;
      }
    }
  }
}

template <typename T, int DH>
__global__ void k_attn_merge(const float* __restrict__ part, int H, int splits, T* __restrict__ o) {
  const int h = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const float* pp = part + ((size_t)b * H + h) * splits * (DH + 2);
  float M = -INFINITY;
  for (int s = 0; s < splits; ++s) M = fmaxf(M, pp[s * (DH + 2)]);
  float L = 0.f, A = 0.f;
  for (int s = 0; s < splits; ++s) {
    const float ms = pp[s * (DH + 2)];
    if (ms == -INFINITY) continue;
    const float f = __expf(ms - M);
    L += pp[s * (DH + 2) + 1] * f;
    A += pp[s * (DH + 2) + 2 + t] * f;
  }
  st<T>(o, (size_t)b * H * DH + h * DH + t, A / L);
}

template <typename T>
static hipError_t decode_t(const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh, int cap, int splits,
                           const float2* rope, void* k, void* v, float* part, void* o, hipStream_t s) {
  const float scale = 1.0f / sqrtf((float)dh);
  const dim3 grid(splits, H, B);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_decode<T, 64>), grid, dim3(64 * decode_waves<64>()), 0, s, qkv, lens, jpos, H, cap, splits, rope, (T*)k,
                       (T*)v, part, (T*)o, scale);
  else
    hipLaunchKernelGGL((k_attn_decode<T, 128>), grid, dim3(64 * decode_waves<128>()), 0, s, qkv, lens, jpos, H, cap, splits, rope, (T*)k,
                       (T*)v, part, (T*)o, scale);
  return hipGetLastError();
}

hipError_t attn_decode(int ct, const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh, int cap,
                       int splits, const float2* rope, void* kslab, void* vslab, float* part, void* o, hipStream_t s) {
  if (ct == DT_F32) return decode_t<float>(qkv, lens, jpos, B, H, dh, cap, splits, rope, kslab, vslab, part, o, s);
  return decode_t<f16>(qkv, lens, jpos, B, H, dh, cap, splits, rope, kslab, vslab, part, o, s);
}

hipError_t attn_merge(int ct, const float* part, int B, int H, int dh, int splits, void* o, hipStream_t s) {
  const dim3 grid(H, B);
  if (ct == DT_F32) {
    if (dh == 64) hipLaunchKernelGGL((k_attn_merge<float, 64>), grid, dim3(64), 0, s, part, H, splits, (float*)o);
    else hipLaunchKernelGGL((k_attn_merge<float, 128>), grid, dim3(128), 0, s, part, H, splits, (float*)o);
  } else {
    if (dh == 64) hipLaunchKernelGGL((k_attn_merge<f16, 64>), grid, dim3(64), 0, s, part, H, splits, (f16*)o);
    else hipLaunchKernelGGL((k_attn_merge<f16, 128>), grid, dim3(128), 0, s, part, H, splits, (f16*)o);
  }
  return hipGetLastError();
}

}  // namespace ams

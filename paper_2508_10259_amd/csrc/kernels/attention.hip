// Attention over the cached context.
//
// K/V of one layer: K and V each a pool of pages [page][head][64][head_dim] in
// the model compute type; row b's position t sits in page pt[b * ppr + t / 64],
// slot t % 64, so the keys of one (row, head) come in contiguous runs of 64.
// Every kernel reads or writes keys in blocks that lie within one or two pages
// and looks their pages up once per block.
//
//  * k_kv_append:     new tokens of a pass -> rotate k (RoPE), write k and v
//                     at their absolute positions.
//  * k_attn_prefill_mfma (fp16) / k_attn_prefill (fp32): causal attention of
//                     a pass's tokens (a row's new segment at positions
//                     pos..pos+n-1) over keys 0..pos+n-1 of that row, K/V
//                     tiles staged in LDS, online softmax; the fp16 kernel
//                     runs both products on MFMA.  k_attn_extend (fp16) takes
//                     passes whose segments are at most 16 tokens long.
//  * k_attn_decode:   one query per row at position p = lens[b] + jpos (a
//                     fed-back action token).  Appends its own K/V, then
//                     each workgroup covers one split of the row's keys 0..p
//                     (split by the actual length, so no workgroup idles on
//                     unused capacity) and each of its waves a block of keys
//                     at a time.  Lanes are laid over (key, 16-byte chunk of
//                     the head dimension) for both K and V, so every load is
//                     row-contiguous; a score is a chunk dot product summed
//                     over the key's lanes with DPP, the online softmax runs
//                     on wavefront shuffles, and each lane keeps the weights
//                     of its own keys for P.V.  The split partials (m, l,
//                     acc) are merged by k_attn_merge with log-sum-exp
//                     weights.
#include "common.h"
#include "kernels.h"

namespace ams {

// Element offset of (page, head h, slot) in one layer's K or V pool.
__device__ __forceinline__ size_t kv_slot(int page, int H, int h, int slot, int dh) {
  return (((size_t)page * H + h) * KV_PAGE + slot) * dh;
}
// Page of row b's position t (t < capacity).
__device__ __forceinline__ int kv_page(const KvPages& kp, int b, int t) { return kp.pt[(size_t)b * kp.ppr + (t >> 6)]; }
// The same at a position that is uniform across the wave (a scalar load).
__device__ __forceinline__ int kv_page_u(const KvPages& kp, int b, int t) {
  return ld_const_uniform(kp.pt, (size_t)__builtin_amdgcn_readfirstlane(b) * kp.ppr + __builtin_amdgcn_readfirstlane(t >> 6));
}

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
                                                   int n_seg, int H, int dh, KvPages kp, const float2* __restrict__ rope,
                                                   T* __restrict__ kslab, T* __restrict__ vslab) {
  const int i = blockIdx.x;
  const int s = find_seg(off, n_seg, i);
  const int b = row[s], p = pos[s] + (i - off[s]);
  const int pg = kv_page(kp, b, p);
  const int d = H * dh, half = dh / 2;
  const float* k = qkv + (size_t)i * 3 * d + d;
  const float* v = k + d;
  for (int e = threadIdx.x; e < H * half; e += blockDim.x) {
    const int h = e / half, ii = e % half;
    const float2 cs = rope[(size_t)p * half + ii];
    const float a = k[h * dh + ii], c = k[h * dh + ii + half];
    T* dst = kslab + kv_slot(pg, H, h, p & (KV_PAGE - 1), dh);
    st<T>(dst, ii, a * cs.x - c * cs.y);
    st<T>(dst, ii + half, a * cs.y + c * cs.x);
  }
  for (int e = threadIdx.x; e < d; e += blockDim.x) {
    const int h = e / dh, dd = e % dh;
    st<T>(vslab + kv_slot(pg, H, h, p & (KV_PAGE - 1), dh), dd, v[e]);
  }
}

// tok_base[t] = element offset of (page, head 0, slot) of the pass's token t
// in a layer's pool, tok_pos[t] = its position (the tables of gemm_qkv_kv)
__global__ __launch_bounds__(256) void k_tok_tables(const int32_t* __restrict__ row, const int32_t* __restrict__ pos,
                                                    const int32_t* __restrict__ off, int n_seg, int n_tok, int H,
                                                    int dh, KvPages kp, int64_t* __restrict__ tok_base,
                                                    int32_t* __restrict__ tok_pos) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_tok) return;
  const int s = find_seg(off, n_seg, t);
  const int b = row[s], p = pos[s] + (t - off[s]);
  tok_base[t] = (int64_t)kv_slot(kv_page(kp, b, p), H, 0, p & (KV_PAGE - 1), dh);
  tok_pos[t] = p;
}

hipError_t tok_tables(Segs sg, KvPages kp, int H, int dh, int64_t* tok_base, int32_t* tok_pos, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_tok_tables, dim3((sg.n_tok + 255) / 256), dim3(256), 0, s, sg.row, sg.pos, sg.off, sg.n_seg,
                     sg.n_tok, H, dh, kp, tok_base, tok_pos);
  return hipGetLastError();
}

// The fp16 append from a pass's token tables (tok_base: element offset of the
// token's (page, head 0, slot), tok_pos: its position): no per-token search of
// the segments and the page table in every layer, and four values per 16-byte
// load; the same arithmetic as k_kv_append, so the same fp16 values.
__global__ __launch_bounds__(256) void k_kv_append_tab(const float* __restrict__ qkv,
                                                       const int64_t* __restrict__ tok_base,
                                                       const int32_t* __restrict__ tok_pos, int H, int dh,
                                                       const float2* __restrict__ rope, f16* __restrict__ kslab,
                                                       f16* __restrict__ vslab) {
  const int i = blockIdx.x;
  const size_t base = (size_t)tok_base[i];
  const int p = tok_pos[i];
  const int d = H * dh, half = dh / 2, hq = half / 4;
  const float* k = qkv + (size_t)i * 3 * d + d;
  const float* v = k + d;
  typedef _Float16 half4v __attribute__((ext_vector_type(4)));
  for (int e = threadIdx.x; e < H * hq; e += blockDim.x) {  // 4 rotation pairs of head h
    const int h = e / hq, ii = 4 * (e % hq);
    const float4 a = *(const float4*)(k + h * dh + ii), c = *(const float4*)(k + h * dh + ii + half);
    const float4 r0 = *(const float4*)(rope + (size_t)p * half + ii), r1 = *(const float4*)(rope + (size_t)p * half + ii + 2);
    const float av[4] = {a.x, a.y, a.z, a.w}, cv[4] = {c.x, c.y, c.z, c.w};
    const float cx[4] = {r0.x, r0.z, r1.x, r1.z}, cy[4] = {r0.y, r0.w, r1.y, r1.w};
    half4v lo, hi;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lo[j] = sat16(av[j] * cx[j] - cv[j] * cy[j]);
      hi[j] = sat16(av[j] * cy[j] + cv[j] * cx[j]);
    }
    f16* dst = kslab + base + (size_t)h * KV_PAGE * dh;
    *(half4v*)(dst + ii) = lo;
    *(half4v*)(dst + ii + half) = hi;
  }
  for (int e = threadIdx.x; e < d / 4; e += blockDim.x) {
    const int h = 4 * e / dh, dd = 4 * e % dh;
    const float4 x = *(const float4*)(v + 4 * e);
    const half4v y = {sat16(x.x), sat16(x.y), sat16(x.z), sat16(x.w)};
    *(half4v*)(vslab + base + (size_t)h * KV_PAGE * dh + dd) = y;
  }
}

hipError_t kv_append_tab(const float* qkv, int n_tok, const int64_t* tok_base, const int32_t* tok_pos, int H, int dh,
                         const float2* rope, void* kslab, void* vslab, hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  if (dh % 8 != 0 || !tok_base || !tok_pos) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_kv_append_tab, dim3(n_tok), dim3(256), 0, s, qkv, tok_base, tok_pos, H, dh, rope, (f16*)kslab,
                     (f16*)vslab);
  return hipGetLastError();
}

hipError_t kv_append(int ct, const float* qkv, Segs sg, int H, int dh, KvPages kp, const float2* rope,
                     void* kslab, void* vslab, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  if (ct == DT_F32)
    hipLaunchKernelGGL(k_kv_append<float>, dim3(sg.n_tok), dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off,
                       sg.n_seg, H, dh, kp, rope, (float*)kslab, (float*)vslab);
  else
    hipLaunchKernelGGL(k_kv_append<f16>, dim3(sg.n_tok), dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off,
                       sg.n_seg, H, dh, kp, rope, (f16*)kslab, (f16*)vslab);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------

template <typename T, int DH>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ qkv, const int32_t* __restrict__ row,
                                                      const int32_t* __restrict__ pos,
                                                      const int32_t* __restrict__ off, int H, KvPages kp,
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
  float m = -INFINITY, l = 0.f, acc[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) acc[i] = 0.f;

  for (int k0 = 0; k0 < kv_end; k0 += KT) {
    __syncthreads();  // Qs ready on the first pass; Ks/Vs/Ps free on later ones
    const size_t tb = kv_slot(kv_page(kp, b, k0), H, h, k0 & (KV_PAGE - 1), DH);  // the tile lies in one page
    for (int e = tid; e < KT * DH; e += blockDim.x) {
      const int kk = e / DH, dd = e % DH;
      const bool ok = k0 + kk < kv_end;
      Ks[kk][dd] = ok ? ld<T>(kslab, tb + (size_t)kk * DH + dd) : 0.f;
      Vs[kk][dd] = ok ? ld<T>(vslab, tb + (size_t)kk * DH + dd) : 0.f;
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

// Sum (max) over each aligned group of N lanes (N <= 32), every lane of a
// group receiving the same total: DPP quad permutes for distances 1 and 2,
// half-row and row mirrors for 4 and 8 (their partner lanes hold equal
// partial results by then), a lane shuffle for 16.  A group of 16 is one DPP
// row, so its reductions take no LDS round trip (ds_bpermute).
template <int CTRL> __device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int N> __device__ __forceinline__ float group_sum(float v) {
  if constexpr (N >= 2) v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
  if constexpr (N >= 4) v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
  if constexpr (N >= 8) v += dpp_mov<0x141>(v);  // row_half_mirror
  if constexpr (N >= 16) v += dpp_mov<0x140>(v); // row_mirror
  if constexpr (N >= 32) v += __shfl_xor(v, 16, 64);
  return v;
}
template <int N> __device__ __forceinline__ float group_max(float v) {
  if constexpr (N >= 2) v = fmaxf(v, dpp_mov<0xB1>(v));
  if constexpr (N >= 4) v = fmaxf(v, dpp_mov<0x4E>(v));
  if constexpr (N >= 8) v = fmaxf(v, dpp_mov<0x141>(v));
  if constexpr (N >= 16) v = fmaxf(v, dpp_mov<0x140>(v));
  if constexpr (N >= 32) v = fmaxf(v, __shfl_xor(v, 16, 64));
  return v;
}

template <int DH>
__global__ __launch_bounds__(256) void k_attn_prefill_mfma(const float* __restrict__ qkv,
                                                           const int32_t* __restrict__ row,
                                                           const int32_t* __restrict__ pos,
                                                           const int32_t* __restrict__ off, int H, KvPages kp,
                                                           const float2* __restrict__ rope,
                                                           const f16* __restrict__ kslab,
                                                           const f16* __restrict__ vslab, f16* __restrict__ o,
                                                           float scale) {
  // LDS row pitches: K rows of DH + 16 halves and V^T rows of KT + 16 (288 / 160
  // bytes) keep the 16-byte fragment reads (lane r reads row r) free of bank
  // conflicts on gfx950, as every pitch of 32 mod 64 bytes does.
  constexpr int QT = 64, KT = 64, HALF = DH / 2, KPAD = DH + 16, VPAD = KT + 16, PPAD = KT + 8;
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

  f16* Pw = Ps + wave * 16 * PPAD;
  constexpr int CH = DH / 8;  // 16-byte chunks per key row

  // A key tile goes global -> registers -> LDS; the next tile's loads are in
  // flight while the current one computes.  K: item c (< KT * CH) is key c / CH,
  // chunk c % CH.  V^T: item c takes keys 4(c & 15) .. +3 of the 16-byte dim
  // chunk c >> 4 and writes, per dim, those 4 keys as one 8-byte word; the 16
  // lanes of a group fill one V^T row (64 keys), which keeps the writes free of
  // bank conflicts.
  constexpr int KI = KT * CH / 256, NV = KT / 4 * CH, VI = (NV + 255) / 256;
  uint4 kreg[KI], vreg[VI][4];
  auto load_tile = [&](int kt) __attribute__((always_inline)) {
    const size_t tb = kv_slot(kv_page_u(kp, b, kt), H, h, 0, DH);  // a 64-key tile is one page
    const f16* Kb = kslab + tb;
    const f16* Vb = vslab + tb;
#pragma unroll
    for (int q = 0; q < KI; ++q) {
      const int c = tid + 256 * q, kk = c / CH, ch = c % CH;
      kreg[q] = kt + kk < kv_end ? *(const uint4*)(Kb + (size_t)kk * DH + ch * 8) : uint4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int q = 0; q < VI; ++q) {
      const int c = tid + 256 * q, kq = c & 15, ch = c >> 4;
      if (c < NV)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kt + 4 * kq + i;
          vreg[q][i] = key < kv_end ? *(const uint4*)(Vb + (size_t)(key - kt) * DH + ch * 8) : uint4{0u, 0u, 0u, 0u};
        }
    }
  };
  load_tile(0);
  // Q fragments: this lane's query row r of the wave, dims 32i + 8g + e (the
  // first key tile's loads are already in flight); rows past the segment read
  // row 0 and are zeroed
  half8 qf[NQI];
  {
    const int qi = q_lo + wave * 16 + r;
    const bool ok = qi < n;
    const float* q = qkv + (size_t)(t0 + (ok ? qi : 0)) * 3 * d + h * DH;
    const float2* rp = rope + (size_t)(p0 + (ok ? qi : 0)) * HALF;
#pragma unroll
    for (int i = 0; i < NQI / 2; ++i) {
      const int d0 = 32 * i + 8 * g;  // < HALF; its partner is d0 + HALF
      float a[8], c[8];
      float2 cs[8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float4 av = *(const float4*)(q + d0 + 4 * u), cv = *(const float4*)(q + d0 + HALF + 4 * u);
        a[4 * u] = av.x; a[4 * u + 1] = av.y; a[4 * u + 2] = av.z; a[4 * u + 3] = av.w;
        c[4 * u] = cv.x; c[4 * u + 1] = cv.y; c[4 * u + 2] = cv.z; c[4 * u + 3] = cv.w;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 t = *(const float4*)(rp + d0 + 2 * u);
        cs[2 * u] = float2{t.x, t.y};
        cs[2 * u + 1] = float2{t.z, t.w};
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ae = ok ? a[e] : 0.f, ce = ok ? c[e] : 0.f;
        qf[i][e] = (f16)((ae * cs[e].x - ce * cs[e].y) * scale);
        qf[i + NQI / 2][e] = (f16)((ae * cs[e].y + ce * cs[e].x) * scale);
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

  for (int kt = 0; kt < kv_end; kt += KT) {
    __syncthreads();  // previous tile's Ks / VT / Ps reads are done
#pragma unroll
    for (int q = 0; q < KI; ++q) {
      const int c = tid + 256 * q, kk = c / CH, ch = c % CH;
      *(uint4*)(Ks + kk * KPAD + ch * 8) = kreg[q];
    }
#pragma unroll
    for (int q = 0; q < VI; ++q) {
      const int c = tid + 256 * q, kq = c & 15, ch = c >> 4;
      if (c < NV) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          typedef _Float16 half4v __attribute__((ext_vector_type(4)));
          const half4v w = {__builtin_bit_cast(half8, vreg[q][0])[e], __builtin_bit_cast(half8, vreg[q][1])[e],
                            __builtin_bit_cast(half8, vreg[q][2])[e], __builtin_bit_cast(half8, vreg[q][3])[e]};
          *(half4v*)(VT + (ch * 8 + e) * VPAD + 4 * kq) = w;
        }
      }
    }
    __syncthreads();
    if (kt + KT < kv_end) load_tile(kt + KT);

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
      v = group_max<16>(v);
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
      rs = group_sum<16>(rs);
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


// Short segments (at most 16 new tokens per row, e.g. a step's observation
// tokens): one workgroup of 4 waves per (segment, head).  The up to 16
// queries are the MFMA M side; the waves split the keys in blocks of 32 (wave
// w takes blocks w, w + 4, ...), each with its own online softmax, and merge
// in LDS at the end.  K fragments come straight from global memory in the B
// layout (one key row per lane group); V goes through a per-wave transposed
// LDS tile: rows of 32 keys (64 bytes, unpadded) whose four 16-byte key chunks
// are swizzled by row (chunk ^ ((row >> 1) & 3)), written as 8-byte words of 4
// keys by lane groups of 8 that fill one row.  On gfx950 that keeps the
// fragment reads free of bank conflicts and the writes near it.
constexpr int EXT_WAVES = 4, EXT_KB = 32;

template <int DH> struct ExtGeo {
  static constexpr int NQI = DH / 32;       // MFMA k-steps of S
  static constexpr int NDJ = DH / 16;       // 16-wide dim blocks of O
  static constexpr int VPAD = EXT_KB;       // V^T tile row (keys), chunks swizzled
  static constexpr int PPAD = EXT_KB + 8;
  static constexpr int VCH = DH / 8;        // 16-byte chunks of a key row
  static constexpr int VLD = EXT_KB * VCH / 64;  // 16-byte V loads per lane per block
  static constexpr int VPASS = VCH / 8;          // passes of 8 dim chunks (4 key rows each)
  static constexpr size_t WAVE_LDS = (size_t)(DH * VPAD + 16 * PPAD) * 2;
};

template <int DH>
__global__ __launch_bounds__(64 * EXT_WAVES, 2) void k_attn_extend(const float* __restrict__ qkv,
                                                                const int32_t* __restrict__ row,
                                                                const int32_t* __restrict__ pos,
                                                                const int32_t* __restrict__ off, int H, KvPages kp,
                                                                const float2* __restrict__ rope,
                                                                const f16* __restrict__ kslab,
                                                                const f16* __restrict__ vslab, f16* __restrict__ o,
                                                                float scale, const int32_t* __restrict__ order) {
  using G = ExtGeo<DH>;
  constexpr int NQI = G::NQI, NDJ = G::NDJ, VPAD = G::VPAD, PPAD = G::PPAD, VLD = G::VLD, VPASS = G::VPASS;
  constexpr int HALF = DH / 2;
  extern __shared__ __attribute__((aligned(16))) unsigned char ext_sm[];
  // segments with the most keys first (order), so the launch does not end on them
  const int sg = order ? __builtin_amdgcn_readfirstlane(order[blockIdx.z]) : (int)blockIdx.z;
  const int h = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int b = row[sg], p0 = pos[sg], t0 = off[sg], n = off[sg + 1] - off[sg];  // n <= 16
  const int d = H * DH;
  const int kv_end = p0 + n;  // keys 0 .. p0+n-1
  f16* VT = (f16*)(ext_sm + wave * G::WAVE_LDS);  // [DH][VPAD]: V^T of this wave's block
  f16* Pw = VT + DH * VPAD;                        // [16][PPAD]: P of this wave's block

  // Q fragments (A layout): query r, dims 32i + 8g + e, rotated and scaled;
  // filled after the first key blocks' loads are issued
  half8 qf[NQI];
  int qp[4];  // positions of this lane's C rows (queries 4g + e); -1 past the segment
#pragma unroll
  for (int e = 0; e < 4; ++e) qp[e] = 4 * g + e < n ? p0 + 4 * g + e : -1;

  // this lane's V chunks of a block: keys 4 * vkq .. +3 of the 16-byte dim
  // chunks vq + 8p (p < VPASS)
  const int vkq = lane & 7, vq = lane >> 3;
  static_assert(4 * VPASS == VLD, "V loads per lane");

  uint4 kc[2][NQI], vc[VLD];
  auto load = [&](int kb, uint4 (&kx)[2][NQI], uint4 (&vx)[VLD]) __attribute__((always_inline)) {
    // a block of EXT_KB = 32 keys starts at a multiple of 32 and lies in one page
    const size_t pb = kv_slot(kv_page_u(kp, b, kb), H, h, 0, DH);
    const f16* Kb = kslab + pb;
    const f16* Vb = vslab + pb;
    // every lane loads from its key's slot of the block's page whether or not the
    // key exists (no branch per load): keys past the segment get score -inf
    // (block), and their values are zeroed here, since P = 0 times a stale
    // slot's bits need not be 0
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int key = kb + 16 * c + r;
#pragma unroll
      for (int i = 0; i < NQI; ++i) kx[c][i] = ld_stream(Kb + (size_t)(key & (KV_PAGE - 1)) * DH + 32 * i + 8 * g);
    }
#pragma unroll
    for (int p = 0; p < VPASS; ++p)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb + 4 * vkq + i;
        const uint4 t = ld_stream(Vb + (size_t)(key & (KV_PAGE - 1)) * DH + (vq + 8 * p) * 8);
        const bool ok = key < kv_end;
        vx[4 * p + i] = uint4{ok ? t.x : 0u, ok ? t.y : 0u, ok ? t.z : 0u, ok ? t.w : 0u};
      }
  };

  float m[4], l[4];
  f32x4 acc[NDJ];
#pragma unroll
  for (int e = 0; e < 4; ++e) { m[e] = -INFINITY; l[e] = 0.f; }
#pragma unroll
  for (int j = 0; j < NDJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // one key block: V^T through LDS, S, online softmax, O += P V
  auto block = [&](int kb, const uint4 (&kx)[2][NQI], const uint4 (&vx)[VLD]) __attribute__((always_inline)) {
    // V^T tile of this block (this wave's LDS only): row = dim, 4 keys per write
#pragma unroll
    for (int p = 0; p < VPASS; ++p) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int R = (vq + 8 * p) * 8 + e;
        // dim e of the 4 keys: 16-bit element e of each loaded chunk, packed in pairs
        uint32_t h[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint4& v = vx[4 * p + i];
          const uint32_t dw = (e >> 1) == 0 ? v.x : (e >> 1) == 1 ? v.y : (e >> 1) == 2 ? v.z : v.w;
          h[i] = (e & 1) ? dw >> 16 : dw & 0xffffu;
        }
        *(uint2*)(VT + R * VPAD + (((vkq >> 1) ^ ((R >> 1) & 3)) * 8) + (vkq & 1) * 4) =
            uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
      }
    }
    // S for the two halves of 16 keys
    f32x4 sc[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      sc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < NQI; ++i)
        sc[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qf[i], __builtin_bit_cast(half8, kx[c][i]), sc[c], 0, 0, 0);
    }
    // causal mask and online softmax per query row 4g+e (its keys sit in the 16 lanes sharing g)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float mx = -INFINITY;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int key = kb + 16 * c + r;
        if (key > qp[e] || key >= kv_end) sc[c][e] = -INFINITY;
        mx = fmaxf(mx, sc[c][e]);
      }
      mx = group_max<16>(mx);
      const float m_new = fmaxf(m[e], mx);
      const float alpha = (m_new == -INFINITY) ? 1.f : __expf(m[e] - m_new);
      float rs = 0.f;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const float pv = (sc[c][e] == -INFINITY) ? 0.f : __expf(sc[c][e] - m_new);
        sc[c][e] = pv;
        rs += pv;
      }
      rs = group_sum<16>(rs);
      l[e] = l[e] * alpha + rs;
      m[e] = m_new;
#pragma unroll
      for (int j = 0; j < NDJ; ++j) acc[j][e] *= alpha;
    }
    // P (C layout) -> LDS [query][key] -> A layout
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) Pw[(4 * g + e) * PPAD + 16 * c + r] = (f16)sc[c][e];
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    const half8 pf = *(const half8*)(Pw + r * PPAD + 8 * g);
#pragma unroll
    for (int j = 0; j < NDJ; ++j) {
      const int R = 16 * j + r;
      const half8 vf = *(const half8*)(VT + R * VPAD + ((g ^ ((R >> 1) & 3)) * 8));
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf, vf, acc[j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // the tile reads are done before the next block overwrites it
    __builtin_amdgcn_wave_barrier();
  };
  // the wave's blocks kb, kb + kstep, ...: the next block's K and V loads are in
  // flight while the current one is computed (two register sets, alternating;
  // the launch bound keeps them within 256 VGPRs, two waves per SIMD: at one wave
  // per SIMD the 7B 64-row extension took 149 us against 114 without prefetch, 105 with)
  const int kstep = EXT_WAVES * EXT_KB;
  uint4 kn[2][NQI], vn[VLD];
  int kb = wave * EXT_KB;
  if (kb < kv_end) load(kb, kc, vc);
  {
    // the query row (rows past the segment read row 0 and are zeroed), 8
    // consecutive dims and their rotation partners as 16-byte loads
    const bool ok = r < n;
    const float* q = qkv + (size_t)(t0 + (ok ? r : 0)) * 3 * d + h * DH;
    const float2* rp = rope + (size_t)(p0 + (ok ? r : 0)) * HALF;
#pragma unroll
    for (int i = 0; i < NQI / 2; ++i) {
      const int d0 = 32 * i + 8 * g;  // < HALF; its partner is d0 + HALF
      float a[8], c[8];
      float2 cs[8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float4 av = *(const float4*)(q + d0 + 4 * u), cv = *(const float4*)(q + d0 + HALF + 4 * u);
        a[4 * u] = av.x; a[4 * u + 1] = av.y; a[4 * u + 2] = av.z; a[4 * u + 3] = av.w;
        c[4 * u] = cv.x; c[4 * u + 1] = cv.y; c[4 * u + 2] = cv.z; c[4 * u + 3] = cv.w;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 t = *(const float4*)(rp + d0 + 2 * u);
        cs[2 * u] = float2{t.x, t.y};
        cs[2 * u + 1] = float2{t.z, t.w};
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ae = ok ? a[e] : 0.f, ce = ok ? c[e] : 0.f;
        qf[i][e] = (f16)((ae * cs[e].x - ce * cs[e].y) * scale);
        qf[i + NQI / 2][e] = (f16)((ae * cs[e].y + ce * cs[e].x) * scale);
      }
    }
  }
  while (kb < kv_end) {
    const int nb = kb + kstep;
    if (nb < kv_end) load(nb, kn, vn);
    block(kb, kc, vc);
    if (nb >= kv_end) break;
    const int nb2 = nb + kstep;
    if (nb2 < kv_end) load(nb2, kc, vc);
    block(nb, kn, vn);
    kb = nb2;
  }

  // merge the waves: per-wave (m, l) per query and O rows through LDS (the V^T tiles are free now)
  __syncthreads();
  float* wm = (float*)ext_sm;                 // [wave][16]
  float* wl = wm + EXT_WAVES * 16;            // [wave][16]
  float* wo = wl + EXT_WAVES * 16;            // [wave][16][DH]
  if (r == 0)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      wm[wave * 16 + 4 * g + e] = m[e];
      wl[wave * 16 + 4 * g + e] = l[e];
    }
#pragma unroll
  for (int j = 0; j < NDJ; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) wo[(wave * 16 + 4 * g + e) * DH + 16 * j + r] = acc[j][e];
  __syncthreads();
  for (int idx = tid; idx < n * DH; idx += 64 * EXT_WAVES) {
    const int q = idx / DH, dd = idx % DH;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < EXT_WAVES; ++w) M = fmaxf(M, wm[w * 16 + q]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < EXT_WAVES; ++w) {
      const float mw = wm[w * 16 + q];
      if (mw == -INFINITY) continue;  // a wave without keys for this query
      const float f = __expf(mw - M);
      L += wl[w * 16 + q] * f;
      A += wo[(w * 16 + q) * DH + dd] * f;
    }
    st<f16>(o + (size_t)(t0 + q) * d + h * DH, dd, A / L);
  }
}

template <int DH> constexpr size_t ext_lds() {
  const size_t tiles = EXT_WAVES * ExtGeo<DH>::WAVE_LDS;
  const size_t merge = (size_t)(2 * EXT_WAVES * 16 + EXT_WAVES * 16 * DH) * 4;
  return tiles > merge ? tiles : merge;
}

template <typename T>
static hipError_t prefill_t(const float* qkv, Segs sg, int H, int dh, KvPages kp, const float2* rope, const void* k,
                            const void* v, void* o, hipStream_t s) {
  const dim3 grid((sg.max_len + 63) / 64, H, sg.n_seg);
  const float scale = 1.0f / sqrtf((float)dh);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_prefill<T, 64>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, kp, rope,
                       (const T*)k, (const T*)v, (T*)o, scale);
  else
    hipLaunchKernelGGL((k_attn_prefill<T, 128>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, kp, rope,
                       (const T*)k, (const T*)v, (T*)o, scale);
  return hipGetLastError();
}

hipError_t attn_prefill(int ct, const float* qkv, Segs sg, int H, int dh, KvPages kp, const float2* rope,
                        const void* kslab, const void* vslab, void* o, hipStream_t s) {
  if (sg.n_tok <= 0) return hipSuccess;
  if (ct == DT_F32) return prefill_t<float>(qkv, sg, H, dh, kp, rope, kslab, vslab, o, s);
  const float scale = 1.0f / sqrtf((float)dh);
  if (sg.max_len <= 16) {  // short segments: keys split over the waves
    const dim3 grid(1, H, sg.n_seg);
    if (dh == 64)
      hipLaunchKernelGGL((k_attn_extend<64>), grid, dim3(64 * EXT_WAVES), ext_lds<64>(), s, qkv, sg.row, sg.pos,
                         sg.off, H, kp, rope, (const f16*)kslab, (const f16*)vslab, (f16*)o, scale, sg.order);
    else
      hipLaunchKernelGGL((k_attn_extend<128>), grid, dim3(64 * EXT_WAVES), ext_lds<128>(), s, qkv, sg.row, sg.pos,
                         sg.off, H, kp, rope, (const f16*)kslab, (const f16*)vslab, (f16*)o, scale, sg.order);
    return hipGetLastError();
  }
  const dim3 grid((sg.max_len + 63) / 64, H, sg.n_seg);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_prefill_mfma<64>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, kp, rope,
                       (const f16*)kslab, (const f16*)vslab, (f16*)o, scale);
  else
    hipLaunchKernelGGL((k_attn_prefill_mfma<128>), grid, dim3(256), 0, s, qkv, sg.row, sg.pos, sg.off, H, kp, rope,
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

// Output element of the decode kernels: fp16 outputs also give their rounding
// error to olo when it is non-NULL.
template <typename T> __device__ __forceinline__ void st_out(T* o, T* olo, size_t i, float v) {
  if constexpr (sizeof(T) == 2) split16(v, o, olo, i);
  else o[i] = v;
}

// Decode lane geometry.  A lane holds one 16-byte chunk (CH elements) of the
// head dimension for one key: NC lanes cover a key, a wave covers KS keys per
// iteration and BK keys per block (IT iterations), so K and V loads are both
// row-contiguous across each group of NC lanes.  Blocks are 2 iterations so
// that the kernel fits 128 VGPRs and two 8-wave workgroups share a CU, one
// computing while the other waits for its keys: at 64 rows of the 7B shape
// (rows of 200-700 keys) that measured 20-25% faster than 8-iteration blocks
// at one workgroup per CU, and 5% at 16 rows of 620 keys.
template <typename T, int DH> struct DecGeo {
  static constexpr int CH = Raw<T>::E;
  static constexpr int NC = DH / CH;
  static constexpr int KS = 64 / NC;
  static constexpr int BK = 2 * KS;
  static constexpr int IT = BK / KS;
};
// at most 8 waves (512 threads) per decode workgroup; a launch may use fewer
constexpr int DECODE_MAX_WAVES = 8;


// Max / sum across the lane groups of size N (values uniform within a group).
template <int N> __device__ __forceinline__ float cross_max(float v) {
#pragma unroll
  for (int o = N; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
template <int N> __device__ __forceinline__ float cross_sum(float v) {
#pragma unroll
  for (int o = N; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <typename T, int DH>
__global__ __launch_bounds__(64 * DECODE_MAX_WAVES, 4) void k_attn_decode(
    const float* __restrict__ qkv, const int32_t* __restrict__ lens, int jpos, int H, KvPages kp, int splits,
    const float2* __restrict__ rope, T* __restrict__ kslab, T* __restrict__ vslab, float* __restrict__ part,
    T* __restrict__ o, T* __restrict__ olo, float scale, QkvParts qp, const int32_t* __restrict__ order) {
  using G = DecGeo<T, DH>;
  constexpr int CH = G::CH, NC = G::NC, KS = G::KS, BK = G::BK, IT = G::IT, HALF = DH / 2;
  __shared__ float wm[DECODE_MAX_WAVES], wl[DECODE_MAX_WAVES], wacc[DECODE_MAX_WAVES][DH];
  __shared__ float qs[3 * DH];  // this head's q, k, v of row b when they come as partial sums
  // order (when given) lists the rows longest first, so the workgroups of long
  // rows are dispatched before those of short ones and the launch does not end
  // waiting on a long row's heads
  const int sp = blockIdx.x, h = blockIdx.y;
  const int b = order ? __builtin_amdgcn_readfirstlane(order[blockIdx.z]) : (int)blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, nw = blockDim.x >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: block loops branch on scalars
  const int ks = lane / NC, dc = lane % NC, i0 = dc * CH;  // this lane: key subgroup, first dimension
  const int d = H * DH;
  const int p = lens[b] + jpos;  // position of this pass's token
  const int T_ = p + 1;          // keys 0..p
  const int chunk = (T_ + splits - 1) / splits;
  const int k0 = sp * chunk < T_ ? sp * chunk : T_;
  const int k1 = (k0 + chunk < T_) ? k0 + chunk : T_;

  // one block: key kb + it*KS + ks of each iteration; slot p is not read (its K/V come from registers).
  // The block's BK <= 64 keys lie in at most two pages, looked up once.  Every lane
  // loads whether or not its key exists (a key past the split or slot p reads 16
  // bytes of this row's query instead), so the loads in flight follow one fixed
  // pattern and the wait before a block covers only its own data; the block
  // replaces those values where they are used.
  const uint4* dummy = (const uint4*)(qkv + (size_t)b * 3 * d);
  auto load_block = [&](int kb, uint4 (&kr)[IT], uint4 (&vr)[IT]) {
    // kb is uniform across the wave: the page indices are scalar loads (scalar cache)
    const int ka = __builtin_amdgcn_readfirstlane(min(kb, k1 - 1) >> 6);
    const int kz = __builtin_amdgcn_readfirstlane(min(kb + BK - 1, k1 - 1) >> 6);
    const int pa = ld_const_uniform(kp.pt, (size_t)b * kp.ppr + ka), pz = ld_const_uniform(kp.pt, (size_t)b * kp.ppr + kz);
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int key = kb + it * KS + ks;
      const bool ok = key < k1 && key != p;
      const size_t e = kv_slot((key >> 6) == ka ? pa : pz, H, h, key & (KV_PAGE - 1), DH) + i0;
      // the address is chosen by a select the compiler cannot see through, so it
      // stays one unconditional load instead of a branch per source
      uint64_t ak = ok ? (uint64_t)(kslab + e) : (uint64_t)dummy;
      uint64_t av = ok ? (uint64_t)(vslab + e) : (uint64_t)dummy;
      asm("" : "+v"(ak), "+v"(av));
      typedef unsigned u32x4g __attribute__((ext_vector_type(4)));
      typedef const u32x4g __attribute__((address_space(1))) gvec;  // global, not flat
      // non-temporal, as ld_stream: each pass reads the cache once
      const u32x4g kx = __builtin_nontemporal_load((gvec*)ak), vx = __builtin_nontemporal_load((gvec*)av);
      kr[it] = uint4{kx[0], kx[1], kx[2], kx[3]};  // what a key that does not exist loaded is never used (see block)
      vr[it] = uint4{vx[0], vx[1], vx[2], vx[3]};
    }
  };
  const int kb0 = k0 + wave * BK;
  uint4 kA[IT], vA[IT], kB[IT], vB[IT];
  load_block(kb0, kA, vA);  // in flight during the prologue

  // this lane's CH dimensions of the rotated, scaled query and of the new
  // token's key and value, rounded to the slab type as every later step reads them
  float q[CH], kn[CH], vn[CH];
  {
    const float* qrow = qkv + (size_t)b * 3 * d + h * DH;
    int kstride = d;  // q, k, v of the head at qrow, qrow + kstride, qrow + 2 kstride
    if (qp.part) {
      // the split-K partial sums of the QKV projection, added in split order and
      // divided by the row's rms as the projection's own reduction would
      float t = 0.f;
      if (qp.ss)
        for (int k = lane; k < qp.nss; k += 64) t += qp.ss[(size_t)b * qp.nss + k];
#pragma unroll
      for (int o_ = 32; o_ > 0; o_ >>= 1) t += __shfl_xor(t, o_, 64);
      const float rr = qp.ss ? 1.0f / sqrtf(t * (1.0f / (float)d) + qp.eps) : 1.f;
      const size_t MN = (size_t)gridDim.z * 3 * d;
      for (int x = tid; x < 3 * DH; x += blockDim.x) {
        const size_t col = (size_t)b * 3 * d + (size_t)(x / DH) * d + h * DH + x % DH;
        float v = 0.f;
        for (int sp_ = 0; sp_ < qp.splits; ++sp_) v += qp.part[sp_ * MN + col];
        qs[x] = v * rr;
      }
      __syncthreads();
      qrow = qs;
      kstride = DH;
    }
    const bool lo = i0 < HALF;  // chunks never straddle the rotation halves
    const int j0 = lo ? i0 : i0 - HALF;
#pragma unroll
    for (int e = 0; e < CH; ++e) {
      const float2 cs = rope[(size_t)p * HALF + j0 + e];
      const float qa = qrow[j0 + e], qc = qrow[j0 + e + HALF];
      const float ka = qrow[kstride + j0 + e], kc = qrow[kstride + j0 + e + HALF];
      const float qr = lo ? qa * cs.x - qc * cs.y : qa * cs.y + qc * cs.x;
      const float kr_ = lo ? ka * cs.x - kc * cs.y : ka * cs.y + kc * cs.x;
      q[e] = qr * scale;
      T t;
      st<T>(&t, 0, kr_);
      kn[e] = ld<T>(&t, 0);
      st<T>(&t, 0, qrow[2 * kstride + i0 + e]);
      vn[e] = ld<T>(&t, 0);
    }
  }
  if (k0 <= p && p < k1 && wave == 0 && ks == 0) {  // the split holding p appends the token
    const int pg = ld_const_uniform(kp.pt, (size_t)b * kp.ppr + __builtin_amdgcn_readfirstlane(p >> 6));
    const size_t ep = kv_slot(pg, H, h, p & (KV_PAGE - 1), DH) + i0;
#pragma unroll
    for (int e = 0; e < CH; ++e) {
      st<T>(kslab + ep, e, kn[e]);
      st<T>(vslab + ep, e, vn[e]);
    }
  }

  float m = -INFINITY, l = 0.f, acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.f;

  // one block of keys: scores, online-softmax rescale, P.V
  auto block = [&](int kb, const uint4 (&kr)[IT], const uint4 (&vr)[IT]) {
    float sc[IT];
    float mx = -INFINITY;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int key = kb + it * KS + ks;
      float kv[CH];
      Raw<T>::cvt(kr[it], kv);
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < CH; ++e) s = fmaf(q[e], key == p ? kn[e] : kv[e], s);
      s = group_sum<NC>(s);
      sc[it] = key < k1 ? s : -INFINITY;
      mx = fmaxf(mx, sc[it]);
    }
    const float m_new = fmaxf(m, cross_max<NC>(mx));  // finite: key kb is valid
    const float alpha = __expf(m - m_new);           // m = -inf on the first block gives 0
    float ps = 0.f;
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[e] *= alpha;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int key = kb + it * KS + ks;
      const float pe = __expf(sc[it] - m_new);  // 0 for masked keys
      ps += pe;
      float vv[CH];
      Raw<T>::cvt(vr[it], vv);
#pragma unroll
      // keys past the split: weight 0 and value 0 (what they loaded may not be finite)
      for (int e = 0; e < CH; ++e) acc[e] = fmaf(pe, key == p ? vn[e] : (key < k1 ? vv[e] : 0.f), acc[e]);
    }
    l = l * alpha + cross_sum<NC>(ps);
    m = m_new;
  };
  // two register sets: the next block's loads are in flight while this one computes
  const int stride = nw * BK;
  // (the scheduling barriers keep each block's arithmetic, and with it the wait
  // for its data, after the next block's loads are issued)
  for (int kb = kb0; kb < k1; kb += 2 * stride) {
    load_block(kb + stride, kB, vB);
    __builtin_amdgcn_sched_barrier(0);
    block(kb, kA, vA);
    load_block(kb + 2 * stride, kA, vA);
    __builtin_amdgcn_sched_barrier(0);
    if (kb + stride < k1) block(kb + stride, kB, vB);
  }
  // sum the key subgroups; lanes of subgroup 0 then hold the wave's partial output
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = cross_sum<NC>(acc[e]);
  if (lane == 0) {
    wm[wave] = m;
    wl[wave] = l;
  }
  if (ks == 0)
#pragma unroll
    for (int e = 0; e < CH; ++e) wacc[wave][i0 + e] = acc[e];
  __syncthreads();
  if (tid < DH) {
    float M = wm[0];
    for (int w = 1; w < nw; ++w) M = fmaxf(M, wm[w]);
    float L = 0.f, Acc = 0.f;
    if (M != -INFINITY) {
      for (int w = 0; w < nw; ++w) {
        const float f = __expf(wm[w] - M);
        L += wl[w] * f;
        Acc += wacc[w][tid] * f;
      }
    }
    if (splits == 1) {
      st_out<T>(o, olo, (size_t)b * d + h * DH + tid, Acc / L);
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
__global__ void k_attn_merge(const float* __restrict__ part, int H, int splits, T* __restrict__ o,
                             T* __restrict__ olo) {
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
  st_out<T>(o, olo, (size_t)b * H * DH + h * DH + t, A / L);
}

template <typename T>
static hipError_t decode_t(const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh, int cap, KvPages kp,
                           int splits,
                           const float2* rope, void* k, void* v, float* part, void* o, void* olo, hipStream_t s,
                           QkvParts qp, const int32_t* order) {
  const float scale = 1.0f / sqrtf((float)dh);
  const dim3 grid(splits, H, B);
  // waves: enough for the longest split (ceil(cap / splits) keys) at one block
  // each, and at least DH threads for the output merge
  const int keys = (cap + splits - 1) / splits;
  const int bk = dh == 64 ? DecGeo<T, 64>::BK : DecGeo<T, 128>::BK;
  int nw = (keys + bk - 1) / bk;
  nw = nw < dh / 64 ? dh / 64 : (nw > DECODE_MAX_WAVES ? DECODE_MAX_WAVES : nw);
  if (dh == 64)
    hipLaunchKernelGGL((k_attn_decode<T, 64>), grid, dim3(64 * nw), 0, s, qkv, lens, jpos, H, kp, splits, rope,
                       (T*)k, (T*)v, part, (T*)o, (T*)olo, scale, qp, order);
  else
    hipLaunchKernelGGL((k_attn_decode<T, 128>), grid, dim3(64 * nw), 0, s, qkv, lens, jpos, H, kp, splits, rope,
                       (T*)k, (T*)v, part, (T*)o, (T*)olo, scale, qp, order);
  return hipGetLastError();
}

hipError_t attn_decode(int ct, const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh, int cap, KvPages kp,
                       int splits, const float2* rope, void* kslab, void* vslab, float* part, void* o, hipStream_t s,
                       void* olo, QkvParts qp, const int32_t* order) {
  if (qp.part && (qp.splits < 1 || (qp.ss && qp.nss < 1))) return hipErrorInvalidValue;
  if (ct == DT_F32) {
    if (olo) return hipErrorInvalidValue;
    return decode_t<float>(qkv, lens, jpos, B, H, dh, cap, kp, splits, rope, kslab, vslab, part, o, nullptr, s, qp,
                           order);
  }
  return decode_t<f16>(qkv, lens, jpos, B, H, dh, cap, kp, splits, rope, kslab, vslab, part, o, olo, s, qp, order);
}

hipError_t attn_merge(int ct, const float* part, int B, int H, int dh, int splits, void* o, hipStream_t s,
                      void* olo) {
  const dim3 grid(H, B);
  if (ct == DT_F32) {
    if (olo) return hipErrorInvalidValue;
    if (dh == 64) hipLaunchKernelGGL((k_attn_merge<float, 64>), grid, dim3(64), 0, s, part, H, splits, (float*)o,
                                     (float*)nullptr);
    else hipLaunchKernelGGL((k_attn_merge<float, 128>), grid, dim3(128), 0, s, part, H, splits, (float*)o,
                            (float*)nullptr);
  } else {
    if (dh == 64) hipLaunchKernelGGL((k_attn_merge<f16, 64>), grid, dim3(64), 0, s, part, H, splits, (f16*)o,
                                     (f16*)olo);
    else hipLaunchKernelGGL((k_attn_merge<f16, 128>), grid, dim3(128), 0, s, part, H, splits, (f16*)o,
                            (f16*)olo);
  }
  return hipGetLastError();
}

}  // namespace ams

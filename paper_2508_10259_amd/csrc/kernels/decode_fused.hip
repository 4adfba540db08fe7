// The whole greedy decode of one step in a single persistent launch (fp16
// compute, up to 8 rows): the action head on the last committed position,
// then for each further action token the feed (argmax + bin embedding), every
// decoder layer over the fed-back tokens (the reused K/V prefix plus the
// appended keys), and the head again.  The method's point is that a step only
// computes the tokens it adds (KV reuse, Sec. 3); at up to 8 rows each of those
// passes is a chain of small dependent GEMVs, so launch and ramp latency, not
// bytes, bound it when every phase is its own kernel.
//
// One workgroup per compute unit (all resident at once), 8 waves each.  The
// phases of a pass are separated by a grid barrier instead of a kernel
// boundary.  The L2s of the eight XCDs are not coherent with each other, so
// every value one workgroup writes for another goes through memory: buffer
// stores and loads with the sc1 cache policy, and the s_waitcnt before a
// workgroup arrives at the barrier makes its stores complete first.  Only the
// packed weights, the RoPE table, the row lengths and the bin embeddings
// (never written during a launch) use plain loads.
//
// Barrier: eight group counters (workgroup i arrives at counter i mod 8); the
// last arrival of a group writes the barrier number into its slot of eight
// replicated flag lines, one line per group, and each workgroup polls its
// group's line until all eight slots have reached it (so no line is both
// polled by every workgroup and hit by atomics).  Spinning is bounded: a wait
// that exceeds its bound sets the error word, which makes every other
// workgroup stop at its next barrier, so the grid always drains.
//
// GEMV phases reuse the decode GEMV's MFMA scheme (weight rows on the M side,
// the up-to-8 tokens' fp16 pairs hi | lo as the 16 B columns, waves splitting
// K in chunks of 128, partial sums meeting in LDS).  Units are 16-row strips
// (32 for gate|up) dealt round-robin to the workgroups; the O and down
// projections split K when they have fewer strips than workgroups, and the
// last of a strip's splits to finish (a counter per strip) adds the partial
// sums in split order, so the result does not depend on arrival order.
#include "common.h"
#include "kernels.h"

namespace ams {

namespace {

typedef unsigned u32x4v __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int CP_SC1 = 16;  // cache-policy bits of a buffer access: sc1

__device__ __forceinline__ Rsrc rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 ldc16(Rsrc r, uint32_t off) {
  const u32x4v v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CP_SC1);
  return uint4{v[0], v[1], v[2], v[3]};
}
__device__ __forceinline__ float ldcf(Rsrc r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, CP_SC1));
}
__device__ __forceinline__ void stcf(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, CP_SC1);
}
__device__ __forceinline__ void stch(Rsrc r, uint32_t off, f16 v) {
  __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), r, off, 0, CP_SC1);
}
__device__ __forceinline__ void stc16(Rsrc r, uint32_t off, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(u32x4v{v.x, v.y, v.z, v.w}, r, off, 0, CP_SC1);
}

__device__ __forceinline__ unsigned ld_agent(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned add_agent(unsigned* p, unsigned v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// this thread's outstanding stores (and loads) are complete
__device__ __forceinline__ void vm_drain() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ half8 as_h8(uint4 v) { return __builtin_bit_cast(half8, v); }
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

}  // namespace

// Words of the synchronisation area (256-byte lines).
constexpr int SYNC_LINE = 64;              // group counter g at g * SYNC_LINE
constexpr int SYNC_FLAG = 9 * SYNC_LINE;   // + r * SYNC_LINE + g: group g's flag, replica r
constexpr int SYNC_ERROR = 17 * SYNC_LINE;
constexpr int SYNC_STRIP = 32 * SYNC_LINE;  // + strip: split-K arrival counters
constexpr unsigned SPIN_LIMIT = 1u << 22;   // polls (about a second or more) before a wait gives up

struct FusedSmem {
  float red[8 * 2 * 256];  // [wave][rb][lane][4] GEMV partial sums
  float wsum[8 * 16];      // [wave][token] RMS statistic partials
  float rstd[16];
  float am[8], al[8];      // attention: per-wave max and sum
  float aacc[8][128];      // attention: per-wave output
  int tok[8];              // feed: argmax per row
  int last;                // split-K: this workgroup finishes the strip
  int stop;                // a barrier wait timed out somewhere
};

// Registers a wave fills for the next phase while it waits at the barrier:
// the weights of its first two batches of GEMV chunks (a[0..7], a[8..15]), or
// the first block of keys (a[0..IT-1]) and values (a[IT..2IT-1]) of its
// attention unit.
struct Prefetch {
  uint4 a[16];
};

// Grid barrier number `gen` (1, 2, ... within a launch), in two halves so
// that a workgroup can issue its next phase's weight loads between them:
// arrive() once every thread's stores are complete, then wait_all().
__device__ void arrive(unsigned* sync, unsigned gen) {
  vm_drain();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned G = gridDim.x, grp = blockIdx.x & 7u;
    const unsigned ngrp = G < 8u ? G : 8u;
    const unsigned ng = (G - grp + 7u) / 8u;  // workgroups in this group
    if (add_agent(sync + grp * SYNC_LINE, 1u) == gen * ng - 1u)
      for (unsigned r = 0; r < ngrp; ++r) st_agent(sync + SYNC_FLAG + r * SYNC_LINE + grp, gen);
  }
}
// Wave 0 polls its group's flag line (lane x reads group x mod 8's slot).
// Returns false once any wait of the launch has timed out.
__device__ bool wait_all(unsigned* sync, unsigned gen, FusedSmem& sm) {
  if (threadIdx.x < 64) {
    const unsigned G = gridDim.x, x = threadIdx.x & 7u;
    const unsigned want = x < G ? gen : 0u;
    const unsigned* flag = sync + SYNC_FLAG + (blockIdx.x & 7u) * SYNC_LINE + x;
    unsigned spins = 0;
    while (!__all(ld_agent(flag) >= want)) {
      if ((++spins & 1023u) == 0 && (spins >= SPIN_LIMIT || ld_agent(sync + SYNC_ERROR) != 0u)) {
        if (threadIdx.x == 0) {
          st_agent(sync + SYNC_ERROR, 1u);
          sm.stop = 1;
        }
        break;
      }
    }
  }
  __syncthreads();
  return sm.stop == 0;
}

// GEMV streaming: a wave covers the K chunks [w0, w1) of its unit in batches
// of CB = 2 / RB chunks (8 uint4 of weights per lane), two batches in flight.
template <int RB> struct GB {
  static constexpr int CB = 2 / RB;
};

__device__ __forceinline__ void wave_chunks(int c0, int c1, int& w0, int& w1) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  w0 = c0 + wave * (c1 - c0) / 8;
  w1 = c0 + (wave + 1) * (c1 - c0) / 8;
}

// W is in MFMA fragment order (frag_pack): the A fragment of rows 16 s .. 16 s + 15
// and columns 128 c + 32 i .. + 31 is 1 KB of contiguous memory at block
// (s * K / 128 + c) * 4 + i, lane l's 16 bytes at l * 16.
template <int RB>
__device__ __forceinline__ void load_w(const f16* W, int K, int n0, int cb, int w1, uint4 (&w)[8]) {
  const int lane = threadIdx.x & 63, nch = K >> 7;
#pragma unroll
  for (int j = 0; j < GB<RB>::CB; ++j) {
    if (cb + j < w1) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const f16* blk = W + (((size_t)((n0 >> 4) + rb) * nch + cb + j) * 4) * 512 + lane * 8;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[(j * RB + rb) * 4 + i] = ld_stream(blk + i * 512);
      }
    }
  }
}

template <int RB>
__device__ __forceinline__ void load_x(Rsrc xr, uint32_t xo, int cb, int w1, uint4 (&x)[8]) {
#pragma unroll
  for (int j = 0; j < GB<RB>::CB; ++j) {
    if (cb + j < w1) {
      const uint32_t kb = (uint32_t)(cb + j) << 7;
#pragma unroll
      for (int i = 0; i < 4; ++i) x[j * 4 + i] = ldc16(xr, xo + (kb + 32u * i) * 2u);
    }
  }
}

template <int RB, bool NRM>
__device__ __forceinline__ void mma_batch(const uint4 (&w)[8], const uint4 (&x)[8], int cb, int w1, f32x4 (&acc)[RB],
                                          float& ss0, float& ss1) {
#pragma unroll
  for (int j = 0; j < GB<RB>::CB; ++j) {
    if (cb + j < w1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (NRM) {
          const half2v* p2 = (const half2v*)&x[j * 4 + i];
          ss0 = __builtin_amdgcn_fdot2(p2[0], p2[0], ss0, false);
          ss1 = __builtin_amdgcn_fdot2(p2[1], p2[1], ss1, false);
          ss0 = __builtin_amdgcn_fdot2(p2[2], p2[2], ss0, false);
          ss1 = __builtin_amdgcn_fdot2(p2[3], p2[3], ss1, false);
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(w[(j * RB + rb) * 4 + i]), as_h8(x[j * 4 + i]),
                                                            acc[rb], 0, 0, 0);
      }
    }
  }
}

// Weights of this wave's first two batches of a unit (the part a GEMV unit
// takes from a Prefetch).
template <int RB>
__device__ __forceinline__ void prefetch_gemv(const f16* W, int K, int n0, int c0, int c1, Prefetch& pf) {
  int w0, w1;
  wave_chunks(c0, c1, w0, w1);
  load_w<RB>(W, K, n0, w0, w1, *(uint4(*)[8])pf.a);
  load_w<RB>(W, K, n0, w0 + GB<RB>::CB, w1, *(uint4(*)[8])(pf.a + 8));
}

// GEMV of one unit: rows n0 .. n0 + 16*RB - 1 of W [N][K] (fp16) over K chunks
// [c0, c1) of 128 for up to 8 tokens, input the fp16 pair x = hi + lo read
// through xr (hi at byte 0, lo at lo_off, each [M][K]); the first two
// batches' weights come from pf when use_pf.  The sums over the waves are left in
// sm.red; NRM also leaves 1/rms of each token (statistic of hi over all of K,
// which the unit must then cover) in sm.rstd.
template <int RB, bool NRM>
__device__ __forceinline__ void gemv_unit(const f16* __restrict__ W, int K, int n0, int c0, int c1, Rsrc xr,
                                          uint32_t lo_off, int M, float eps, FusedSmem& sm, Prefetch& pf,
                                          bool use_pf) {
  constexpr int CB = GB<RB>::CB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  int w0, w1;
  wave_chunks(c0, c1, w0, w1);
  f32x4 acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // B column r: token r & 7, hi for r < 8 and lo above; tokens >= M read token 0
  // (their columns are never stored)
  const int tk = r & 7;
  const uint32_t xo = (r >= 8 ? lo_off : 0u) + (uint32_t)(((tk < M ? tk : 0) * K + g * 8) * 2);
  float ss0 = 0.f, ss1 = 0.f;
  // the two stream buffers are the prefetch registers: batches alternate between them
  uint4(&wa)[8] = *(uint4(*)[8])pf.a;
  uint4(&wb)[8] = *(uint4(*)[8])(pf.a + 8);
  uint4 xa[8], xb[8];
  if (!use_pf) {
    load_w<RB>(W, K, n0, w0, w1, wa);
    load_w<RB>(W, K, n0, w0 + CB, w1, wb);
  }
  load_x<RB>(xr, xo, w0, w1, xa);
  load_x<RB>(xr, xo, w0 + CB, w1, xb);
  for (int cb = w0; cb < w1; cb += 2 * CB) {
    mma_batch<RB, NRM>(wa, xa, cb, w1, acc, ss0, ss1);
    if (cb + 2 * CB < w1) {
      load_w<RB>(W, K, n0, cb + 2 * CB, w1, wa);
      load_x<RB>(xr, xo, cb + 2 * CB, w1, xa);
    }
    if (cb + CB < w1) {
      mma_batch<RB, NRM>(wb, xb, cb + CB, w1, acc, ss0, ss1);
      if (cb + 3 * CB < w1) {
        load_w<RB>(W, K, n0, cb + 3 * CB, w1, wb);
        load_x<RB>(xr, xo, cb + 3 * CB, w1, xb);
      }
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) sm.red[((wave * RB + rb) * 64 + lane) * 4 + i] = acc[rb][i];
  if constexpr (NRM) {
    float ss = ss0 + ss1;
    ss += __shfl_xor(ss, 16, 64);
    ss += __shfl_xor(ss, 32, 64);
    if (lane < 16) sm.wsum[wave * 16 + lane] = ss;
  }
  __syncthreads();
  if constexpr (NRM) {
    if (threadIdx.x < 16) {
      float t = 0.f;
      for (int w = 0; w < 8; ++w) t += sm.wsum[w * 16 + threadIdx.x];
      sm.rstd[threadIdx.x] = 1.0f / sqrtf(t / (float)K + eps);
    }
    __syncthreads();
  }
}

// Sum over the waves and over the hi / lo columns of value (rb, ln, i): packed
// row n0 + rb*16 + 4*(ln >> 4) + i, token ln & 15 (< 8).
template <int RB>
__device__ __forceinline__ float gemv_value(const FusedSmem& sm, int rb, int ln, int i) {
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < 8; ++w)
    t += sm.red[((w * RB + rb) * 64 + ln) * 4 + i] + sm.red[((w * RB + rb) * 64 + ln + 8) * 4 + i];
  return t;
}

struct FusedArgs {
  // packed model in MFMA fragment order (per-layer byte strides)
  const f16* wqkv; size_t s_qkv;
  const f16* wo; size_t s_o;
  const f16* wgu; size_t s_gu;
  const f16* wd; size_t s_d;
  const f16* whead;      // [nbp][d], fragment order like the layers' matrices
  const f16* bin_embed;  // [n_bins][d]
  int L, d, H, F, nbp, n_bins;
  float eps, scale;
  // context
  int M, cap, A;
  int split_o, split_d;  // K splits of the O and down projections
  int split_a;           // key splits of the attention
  const int32_t* lens;
  const float2* rope;
  f16* kv; size_t slab;  // K page pool of layer l at kv + 2l*slab elements, V at (2l+1)*slab
  const int32_t* pt; int ppr;  // row b's position t: page pt[b * ppr + t / 64], slot t % 64
  float* h;              // [M][d] residual stream
  f16* hp;               // [2][M][d] its fp16 pair
  const f16* hl; uint32_t hl_lo;  // pair of the last committed position (hi, lo at +hl_lo bytes)
  float* qkv;            // [M][3d]
  f16* op;               // [2][M][d] attention output pair
  f16* ap;               // [2][M][F] SwiGLU output pair
  float* logits;         // [M][nbp]
  float* part;           // split-K partial sums [unit][8][16]
  unsigned* sync;
  unsigned* status;      // host-visible word: set to 1 when a barrier wait gives up (or NULL)
  int32_t* out_tok;      // [M][A]
  float* out_logits;     // [M][A][n_bins] or NULL
  const int32_t* forced; // [M][A] or NULL
};

__device__ __forceinline__ const f16* layer_w(const f16* base, size_t stride, int l) {
  return (const f16*)((const char*)base + (size_t)l * stride);
}

// GEMV phases ------------------------------------------------------------------

// y = W x * rstd (x the pair read through xr), stored fp32 at out[tok*ldo + n]
// (sc1); j_head >= 0 (the head) also writes the caller's out_logits for bins < n_bins.
__device__ void phase_store(const FusedArgs& a, const f16* W, int N, int K, Rsrc xr, uint32_t lo_off, Rsrc outr,
                            int ldo, int j_head, FusedSmem& sm, Prefetch& pf) {
  const int units = N / 16;
  for (int u = blockIdx.x; u < units; u += gridDim.x) {
    gemv_unit<1, true>(W, K, u * 16, 0, K >> 7, xr, lo_off, a.M, a.eps, sm, pf, u == (int)blockIdx.x);
    if (threadIdx.x < 256) {
      const int ln = threadIdx.x >> 2, i = threadIdx.x & 3, tok = ln & 15;
      if (tok < 8 && tok < a.M) {
        const int n = u * 16 + 4 * (ln >> 4) + i;
        const float y = gemv_value<1>(sm, 0, ln, i) * sm.rstd[tok];
        stcf(outr, (uint32_t)(tok * ldo + n) * 4u, y);
        if (j_head >= 0 && a.out_logits && n < a.n_bins)
          a.out_logits[((size_t)tok * a.A + j_head) * a.n_bins + n] = y;
      }
    }
    __syncthreads();
  }
}
__device__ __forceinline__ void prefetch_store(const f16* W, int N, int K, Prefetch& pf) {
  if ((int)blockIdx.x < N / 16) prefetch_gemv<1>(W, K, blockIdx.x * 16, 0, K >> 7, pf);
}

// a = silu(gate) * up of the packed gate|up rows (32-row units), as an fp16 pair.
__device__ void phase_swiglu(const FusedArgs& a, const f16* W, Rsrc xr, uint32_t lo_off, FusedSmem& sm,
                             Prefetch& pf) {
  const int F = a.F, units = (2 * F) / 32;
  const Rsrc apr = rsrc(a.ap, (uint32_t)(2 * a.M * F * 2));
  const uint32_t alo = (uint32_t)(a.M * F * 2);
  for (int u = blockIdx.x; u < units; u += gridDim.x) {
    gemv_unit<2, true>(W, a.d, u * 32, 0, a.d >> 7, xr, lo_off, a.M, a.eps, sm, pf, u == (int)blockIdx.x);
    if (threadIdx.x < 256) {
      const int ln = threadIdx.x >> 2, i = threadIdx.x & 3, tok = ln & 15;
      if (tok < 8 && tok < a.M) {
        const float sc = sm.rstd[tok];
        const float gt = gemv_value<2>(sm, 0, ln, i) * sc, up = gemv_value<2>(sm, 1, ln, i) * sc;
        const float v = silu(gt) * up;
        const f16 hi = sat16(v), lo = sat16(v - (float)hi);
        const uint32_t o = (uint32_t)(tok * F + u * 16 + 4 * (ln >> 4) + i) * 2u;
        stch(apr, o, hi);
        stch(apr, alo + o, lo);
      }
    }
    __syncthreads();
  }
}
__device__ __forceinline__ void prefetch_swiglu(const FusedArgs& a, const f16* W, Prefetch& pf) {
  if ((int)blockIdx.x < (2 * a.F) / 32) prefetch_gemv<2>(W, a.d, blockIdx.x * 32, 0, a.d >> 7, pf);
}

// h += W x (x the pair read through xr, K = its width), K split S ways when
// the strips are few; writes h and its fp16 pair.
__device__ void phase_resid(const FusedArgs& a, const f16* W, int K, int S, Rsrc xr, uint32_t lo_off, FusedSmem& sm,
                            Prefetch& pf) {
  const int d = a.d, strips = d / 16, units = strips * S, nch = K >> 7;
  const Rsrc hr = rsrc(a.h, (uint32_t)(a.M * d * 4));
  const Rsrc hpr = rsrc(a.hp, (uint32_t)(2 * a.M * d * 2));
  const Rsrc pr = rsrc(a.part, (uint32_t)(units * 8 * 16 * 4));
  const uint32_t hlo = (uint32_t)(a.M * d * 2);
  for (int u = blockIdx.x; u < units; u += gridDim.x) {
    const int strip = u / S, sp = u % S;
    const int ln = threadIdx.x >> 2, i = threadIdx.x & 3, tok = ln & 15, row = 4 * (ln >> 4) + i;
    const bool ok = threadIdx.x < 256 && tok < 8 && tok < a.M;
    // this thread's residual value, written two phases ago: its load overlaps the GEMV
    const uint32_t e = (uint32_t)(tok * d + strip * 16 + row);
    const float h_old = ok ? ldcf(hr, e * 4u) : 0.f;
    gemv_unit<1, false>(W, K, strip * 16, sp * nch / S, (sp + 1) * nch / S, xr, lo_off, a.M, 0.f, sm, pf,
                        u == (int)blockIdx.x);
    float y = ok ? gemv_value<1>(sm, 0, ln, i) : 0.f;
    bool fin = true;
    if (S > 1) {
      if (ok) stcf(pr, (uint32_t)((u * 8 + tok) * 16 + row) * 4u, y);
      vm_drain();
      __syncthreads();
      if (threadIdx.x == 0) {
        unsigned* cnt = a.sync + SYNC_STRIP + strip;
        const bool last = add_agent(cnt, 1u) == (unsigned)(S - 1);
        if (last) st_agent(cnt, 0u);  // every split has arrived: reset for the next phase
        sm.last = last;
      }
      __syncthreads();
      fin = sm.last != 0;
      if (fin && ok) {  // all partials requested at once, added in split order
        float ps[FUSED_MAX_SPLIT];
#pragma unroll
        for (int s = 0; s < FUSED_MAX_SPLIT; ++s)
          ps[s] = s < S ? ldcf(pr, (uint32_t)(((strip * S + s) * 8 + tok) * 16 + row) * 4u) : 0.f;
        y = 0.f;
#pragma unroll
        for (int s = 0; s < FUSED_MAX_SPLIT; ++s)
          if (s < S) y += ps[s];
      }
    }
    if (fin && ok) {
      const float hn = h_old + y;
      stcf(hr, e * 4u, hn);
      const f16 hi = sat16(hn);
      stch(hpr, e * 2u, hi);
      stch(hpr, hlo + e * 2u, sat16(hn - (float)hi));
    }
    __syncthreads();
  }
}
__device__ __forceinline__ void prefetch_resid(const FusedArgs& a, const f16* W, int K, int S, Prefetch& pf) {
  const int u = blockIdx.x, nch = K >> 7;
  if (u < (a.d / 16) * S) {
    const int strip = u / S, sp = u % S;
    prefetch_gemv<1>(W, K, strip * 16, sp * nch / S, (sp + 1) * nch / S, pf);
  }
}

// Attention phase ------------------------------------------------------------

template <int DH> struct FGeo {
  static constexpr int CH = 8;           // fp16 elements per 16-byte chunk
  static constexpr int NC = DH / CH;     // lanes per key
  static constexpr int KS = 64 / NC;     // keys per wave per iteration
  static constexpr int IT = DH == 64 ? 5 : 8;  // iterations per block: all 8 waves busy on ~300 keys at 64
  static constexpr int BK = KS * IT;     // keys per wave per block
};

template <int N> __device__ __forceinline__ float fdpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), N, 0xF, 0xF, false));
}
template <int N> __device__ __forceinline__ float fgroup_sum(float v) {
  if constexpr (N >= 2) v += fdpp<0xB1>(v);
  if constexpr (N >= 4) v += fdpp<0x4E>(v);
  if constexpr (N >= 8) v += fdpp<0x141>(v);
  if constexpr (N >= 16) v += fdpp<0x140>(v);
  if constexpr (N >= 32) v += __shfl_xor(v, 16, 64);
  return v;
}
template <int N> __device__ __forceinline__ float fcross_max(float v) {
#pragma unroll
  for (int o = N; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
template <int N> __device__ __forceinline__ float fcross_sum(float v) {
#pragma unroll
  for (int o = N; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Keys of split sp of S over positions 0..p: [k0, k1).
__device__ __forceinline__ void key_range(int p, int sp, int S, int& k0, int& k1) {
  const int T_ = p + 1, ch = (T_ + S - 1) / S;
  k0 = sp * ch < T_ ? sp * ch : T_;
  k1 = k0 + ch < T_ ? k0 + ch : T_;
}

// Byte offset of (row b's position t, head h, dimension i0) in a layer's K or V
// page pool, given t's page.
template <int DH>
__device__ __forceinline__ uint32_t kv_off(int page, int H, int h, int t, int i0) {
  return ((((uint32_t)page * H + h) * 64u + (uint32_t)(t & 63)) * DH + i0) * 2u;
}

// One block of keys kb + it*KS + ks (it < IT) of row b, head h (kb < k1): K into
// kv[0..IT), V into kv[IT..2IT); keys >= k1 and the pass's own position p (its
// K/V come from registers) read zeros.  The block's BK <= 64 keys lie in at most
// two pages, looked up once.
template <int DH>
__device__ __forceinline__ void attn_block(const FusedArgs& a, Rsrc kr, Rsrc vr, int b, int h, int kb, int k1, int p,
                                           uint4 (&kv)[16]) {
  using G = FGeo<DH>;
  const int lane = threadIdx.x & 63, ks = lane / G::NC, i0 = (lane % G::NC) * G::CH;
  // kb and b are uniform across the wave: the page indices are scalar loads (scalar cache)
  const size_t r = (size_t)__builtin_amdgcn_readfirstlane(b) * a.ppr;
  const int ka = __builtin_amdgcn_readfirstlane(kb >> 6);
  const int kz = __builtin_amdgcn_readfirstlane(min(kb + G::BK - 1, k1 - 1) >> 6);
  const int pa = ld_const_uniform(a.pt, r + ka), pz = ld_const_uniform(a.pt, r + kz);
#pragma unroll
  for (int it = 0; it < G::IT; ++it) {
    const int key = kb + it * G::KS + ks;
    const bool ok = key < k1 && key != p;
    const uint32_t off = kv_off<DH>((key >> 6) == ka ? pa : pz, a.H, h, key, i0);
    kv[it] = ok ? ldc16(kr, off) : uint4{0u, 0u, 0u, 0u};
    kv[G::IT + it] = ok ? ldc16(vr, off) : uint4{0u, 0u, 0u, 0u};
  }
}

template <int DH>
__device__ __forceinline__ void prefetch_attn(const FusedArgs& a, int l, int jpos, Prefetch& pf) {
  const int u = blockIdx.x, S = a.split_a;
  if (u >= a.M * a.H * S) return;
  const int item = u / S, sp = u % S, b = item / a.H, h = item % a.H, wave = threadIdx.x >> 6;
  const int p = a.lens[b] + jpos;
  int k0, k1;
  key_range(p, sp, S, k0, k1);
  const int kb0 = k0 + wave * FGeo<DH>::BK;
  if (kb0 >= k1) return;
  const Rsrc kr = rsrc(a.kv + (size_t)(2 * l) * a.slab, (uint32_t)(a.slab * 2));
  const Rsrc vr = rsrc(a.kv + (size_t)(2 * l + 1) * a.slab, (uint32_t)(a.slab * 2));
  attn_block<DH>(a, kr, vr, b, h, kb0, k1, p, pf.a);
}

// One query per (row, head) at position p = lens[b] + jpos over keys 0..p, the
// keys cut into S splits (one unit each): rotates q and the new key, the split
// holding p appends the new K/V there, online softmax over the split's keys
// (lanes over (key, 16-byte chunk of the head), 8 waves).  With S > 1 the
// partials (max, sum, weighted values) meet through memory and the last split
// to finish merges them in split order; the output is an fp16 pair.  The
// first unit's first key block comes from pf.
template <int DH>
__device__ void phase_attn(const FusedArgs& a, int l, int jpos, FusedSmem& sm, Prefetch& pf) {
  using G = FGeo<DH>;
  constexpr int CH = G::CH, NC = G::NC, KS = G::KS, BK = G::BK, IT = G::IT, HALF = DH / 2;
  const int H = a.H, d = a.d, S = a.split_a, units = a.M * H * S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ks = lane / NC, dc = lane % NC, i0 = dc * CH;
  const Rsrc kr_ = rsrc(a.kv + (size_t)(2 * l) * a.slab, (uint32_t)(a.slab * 2));
  const Rsrc vr_ = rsrc(a.kv + (size_t)(2 * l + 1) * a.slab, (uint32_t)(a.slab * 2));
  const Rsrc qr = rsrc(a.qkv, (uint32_t)(a.M * 3 * d * 4));
  const Rsrc opr = rsrc(a.op, (uint32_t)(2 * a.M * d * 2));
  const Rsrc pr = rsrc(a.part, (uint32_t)(units * (DH + 2) * 4));
  const uint32_t olo = (uint32_t)(a.M * d * 2);
  for (int u = blockIdx.x; u < units; u += gridDim.x) {
    const int item = u / S, sp = u % S, b = item / H, h = item % H;
    const int p = a.lens[b] + jpos;
    int k0, k1;
    key_range(p, sp, S, k0, k1);
    const int kb0 = k0 + wave * BK;
    uint4(&kv)[16] = pf.a;  // the first unit's first block was prefetched into these
    if (u != (int)blockIdx.x && kb0 < k1) attn_block<DH>(a, kr_, vr_, b, h, kb0, k1, p, kv);

    // this lane's CH dimensions of the rotated, scaled query and of the new key
    // and value, rounded to fp16 as the slab holds them
    float q[CH], kn[CH], vn[CH];
    {
      const uint32_t qrow = (uint32_t)(b * 3 * d + h * DH);
      const bool lo = i0 < HALF;
      const int j0 = lo ? i0 : i0 - HALF;
      uint4 raw[10];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        raw[c] = ldc16(qr, (qrow + j0 + 4 * c) * 4u);
        raw[2 + c] = ldc16(qr, (qrow + j0 + HALF + 4 * c) * 4u);
        raw[4 + c] = ldc16(qr, (qrow + d + j0 + 4 * c) * 4u);
        raw[6 + c] = ldc16(qr, (qrow + d + j0 + HALF + 4 * c) * 4u);
        raw[8 + c] = ldc16(qr, (qrow + 2 * d + i0 + 4 * c) * 4u);
      }
      const float* f = (const float*)raw;  // qa[8] qc[8] ka[8] kc[8] v[8]
#pragma unroll
      for (int e = 0; e < CH; ++e) {
        const float2 cs = a.rope[(size_t)p * HALF + j0 + e];
        const float qa = f[e], qc = f[8 + e], ka = f[16 + e], kc = f[24 + e];
        const float qrot = lo ? qa * cs.x - qc * cs.y : qa * cs.y + qc * cs.x;
        const float krot = lo ? ka * cs.x - kc * cs.y : ka * cs.y + kc * cs.x;
        q[e] = qrot * a.scale;
        kn[e] = (float)sat16(krot);
        vn[e] = (float)sat16(f[32 + e]);
      }
    }
    if (k0 <= p && p < k1 && wave == 0 && ks == 0) {  // the split holding p appends the token's K and V
      half8 kh, vh;
#pragma unroll
      for (int e = 0; e < CH; ++e) {
        kh[e] = (f16)kn[e];
        vh[e] = (f16)vn[e];
      }
      const int pg = ld_const_uniform(a.pt, (size_t)__builtin_amdgcn_readfirstlane(b) * a.ppr +
                                                __builtin_amdgcn_readfirstlane(p >> 6));
      const uint32_t off = kv_off<DH>(pg, H, h, p, i0);
      stc16(kr_, off, __builtin_bit_cast(uint4, kh));
      stc16(vr_, off, __builtin_bit_cast(uint4, vh));
    }

    float m = -INFINITY, ls = 0.f, acc[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[e] = 0.f;
    for (int kb = kb0; kb < k1; kb += 8 * BK) {
      if (kb != kb0) attn_block<DH>(a, kr_, vr_, b, h, kb, k1, p, kv);
      float sc[IT];
      float mx = -INFINITY;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int key = kb + it * KS + ks;
        const half8 k8 = as_h8(kv[it]);
        float s_ = 0.f;
#pragma unroll
        for (int e = 0; e < CH; ++e) s_ = fmaf(q[e], key == p ? kn[e] : (float)k8[e], s_);
        s_ = fgroup_sum<NC>(s_);
        sc[it] = key < k1 ? s_ : -INFINITY;
        mx = fmaxf(mx, sc[it]);
      }
      const float m_new = fmaxf(m, fcross_max<NC>(mx));
      const float alpha = __expf(m - m_new);
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < CH; ++e) acc[e] *= alpha;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int key = kb + it * KS + ks;
        const float pe = __expf(sc[it] - m_new);
        ps += pe;
        const half8 v8 = as_h8(kv[IT + it]);
#pragma unroll
        for (int e = 0; e < CH; ++e) acc[e] = fmaf(pe, key == p ? vn[e] : (float)v8[e], acc[e]);
      }
      ls = ls * alpha + fcross_sum<NC>(ps);
      m = m_new;
    }
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[e] = fcross_sum<NC>(acc[e]);
    if (lane == 0) {
      sm.am[wave] = m;
      sm.al[wave] = ls;
    }
    if (ks == 0)
#pragma unroll
      for (int e = 0; e < CH; ++e) sm.aacc[wave][i0 + e] = acc[e];
    __syncthreads();
    // this split's (max, sum, weighted values) over its waves
    float Mx = -INFINITY, L = 0.f, Acc = 0.f;
    if (tid < DH) {
      for (int w = 0; w < 8; ++w) Mx = fmaxf(Mx, sm.am[w]);
      if (Mx != -INFINITY) {
        for (int w = 0; w < 8; ++w) {
          if (sm.am[w] == -INFINITY) continue;  // a wave without keys
          const float fw = __expf(sm.am[w] - Mx);
          L += sm.al[w] * fw;
          Acc += sm.aacc[w][tid] * fw;
        }
      }
    }
    bool fin = true;
    if (S > 1) {
      if (tid < DH) {
        const uint32_t base = (uint32_t)u * (DH + 2);
        stcf(pr, (base + 2 + tid) * 4u, Acc);
        if (tid == 0) {
          stcf(pr, base * 4u, Mx);
          stcf(pr, (base + 1) * 4u, L);
        }
      }
      vm_drain();
      __syncthreads();
      if (tid == 0) {
        unsigned* cnt = a.sync + SYNC_STRIP + item;
        const bool last = add_agent(cnt, 1u) == (unsigned)(S - 1);
        if (last) st_agent(cnt, 0u);
        sm.last = last;
      }
      __syncthreads();
      fin = sm.last != 0;
      if (fin && tid < DH) {  // merge the splits in order, every partial requested at once
        const uint32_t b0 = (uint32_t)(item * S) * (DH + 2);
        float pm[FUSED_MAX_ATTN_SPLIT], pl[FUSED_MAX_ATTN_SPLIT], pa[FUSED_MAX_ATTN_SPLIT];
#pragma unroll
        for (int s_ = 0; s_ < FUSED_MAX_ATTN_SPLIT; ++s_) {
          const uint32_t bs = b0 + s_ * (DH + 2);
          pm[s_] = s_ < S ? ldcf(pr, bs * 4u) : -INFINITY;
          pl[s_] = s_ < S ? ldcf(pr, (bs + 1) * 4u) : 0.f;
          pa[s_] = s_ < S ? ldcf(pr, (bs + 2 + tid) * 4u) : 0.f;
        }
        Mx = -INFINITY;
#pragma unroll
        for (int s_ = 0; s_ < FUSED_MAX_ATTN_SPLIT; ++s_) Mx = fmaxf(Mx, pm[s_]);
        L = 0.f;
        Acc = 0.f;
#pragma unroll
        for (int s_ = 0; s_ < FUSED_MAX_ATTN_SPLIT; ++s_) {
          if (pm[s_] == -INFINITY) continue;  // a split without keys (or beyond S)
          const float fw = __expf(pm[s_] - Mx);
          L += pl[s_] * fw;
          Acc += pa[s_] * fw;
        }
      }
    }
    if (fin && tid < DH) {
      const float v = Acc / L;
      const f16 hi = sat16(v);
      const uint32_t o = (uint32_t)(b * d + h * DH + tid) * 2u;
      stch(opr, o, hi);
      stch(opr, olo + o, sat16(v - (float)hi));
    }
    __syncthreads();
  }
}

// Feed phase: argmax of each row's bin logits (lowest bin on ties) -> out_tok
// (workgroup 0); with feed, h and its pair = the bin embedding of the argmax
// or of the clamped forced token, spread over the workgroups.
__device__ void phase_feed(const FusedArgs& a, int j, bool feed, FusedSmem& sm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const Rsrc lr = rsrc(a.logits, (uint32_t)(a.M * a.nbp * 4));
  if (wave < a.M) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int bin = lane; bin < a.n_bins; bin += 64) {
      const float v = ldcf(lr, (uint32_t)(wave * a.nbp + bin) * 4u);
      if (v > bv) { bv = v; bi = bin; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    if (bi < 0 || bi >= a.n_bins) bi = 0;  // every logit NaN
    if (lane == 0) sm.tok[wave] = bi;
  }
  __syncthreads();
  if (blockIdx.x == 0 && (int)threadIdx.x < a.M) a.out_tok[(size_t)threadIdx.x * a.A + j] = sm.tok[threadIdx.x];
  if (!feed) return;
  const int d = a.d;
  const Rsrc hr = rsrc(a.h, (uint32_t)(a.M * d * 4));
  const Rsrc hpr = rsrc(a.hp, (uint32_t)(2 * a.M * d * 2));
  const uint32_t hlo = (uint32_t)(a.M * d * 2);
  for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < a.M * d; idx += gridDim.x * blockDim.x) {
    const int b = idx / d, i = idx % d;
    int t = a.forced ? a.forced[(size_t)b * a.A + j] : sm.tok[b];
    t = t < 0 ? 0 : (t >= a.n_bins ? a.n_bins - 1 : t);
    const f16 e = a.bin_embed[(size_t)t * d + i];
    stcf(hr, (uint32_t)idx * 4u, (float)e);
    stch(hpr, (uint32_t)idx * 2u, e);
    stch(hpr, hlo + (uint32_t)idx * 2u, (f16)0.f);
  }
}

template <int DH>
__global__ __launch_bounds__(512) void k_decode_fused(FusedArgs a) {
  __shared__ FusedSmem sm;
  if (threadIdx.x == 0) sm.stop = 0;
  __syncthreads();
  const int d = a.d, M = a.M;
  unsigned gen = 0;
  Prefetch pf;
  const Rsrc hlr = rsrc(a.hl, a.hl_lo + (uint32_t)(M * d * 2));
  const Rsrc hpr = rsrc(a.hp, (uint32_t)(2 * M * d * 2));
  const Rsrc opr = rsrc(a.op, (uint32_t)(2 * M * d * 2));
  const Rsrc apr = rsrc(a.ap, (uint32_t)(2 * M * a.F * 2));
  const Rsrc qkvr = rsrc(a.qkv, (uint32_t)(M * 3 * d * 4));
  const Rsrc logr = rsrc(a.logits, (uint32_t)(M * a.nbp * 4));
  const uint32_t hlo = (uint32_t)(M * d * 2), olo = hlo, alo = (uint32_t)(M * a.F * 2);
#define AMS_SYNC(PREFETCH)                        \
  do {                                            \
    arrive(a.sync, ++gen);                        \
    PREFETCH;                                     \
    if (!wait_all(a.sync, gen, sm)) goto failed;  \
  } while (0)

  prefetch_store(a.whead, a.nbp, d, pf);
  phase_store(a, a.whead, a.nbp, d, hlr, a.hl_lo, logr, a.nbp, 0, sm, pf);
  for (int j = 1; j < a.A; ++j) {
    AMS_SYNC((void)0);
    phase_feed(a, j - 1, true, sm);
    AMS_SYNC(prefetch_store(layer_w(a.wqkv, a.s_qkv, 0), 3 * d, d, pf));
    for (int l = 0; l < a.L; ++l) {
      const f16* wqkv = layer_w(a.wqkv, a.s_qkv, l);
      const f16* wo = layer_w(a.wo, a.s_o, l);
      const f16* wgu = layer_w(a.wgu, a.s_gu, l);
      const f16* wd = layer_w(a.wd, a.s_d, l);
      phase_store(a, wqkv, 3 * d, d, hpr, hlo, qkvr, 3 * d, -1, sm, pf);
      AMS_SYNC(prefetch_attn<DH>(a, l, j - 1, pf));
      phase_attn<DH>(a, l, j - 1, sm, pf);
      AMS_SYNC(prefetch_resid(a, wo, d, a.split_o, pf));
      phase_resid(a, wo, d, a.split_o, opr, olo, sm, pf);
      AMS_SYNC(prefetch_swiglu(a, wgu, pf));
      phase_swiglu(a, wgu, hpr, hlo, sm, pf);
      AMS_SYNC(prefetch_resid(a, wd, a.F, a.split_d, pf));
      phase_resid(a, wd, a.F, a.split_d, apr, alo, sm, pf);
      if (l + 1 < a.L) AMS_SYNC(prefetch_store(layer_w(a.wqkv, a.s_qkv, l + 1), 3 * d, d, pf));
      else AMS_SYNC(prefetch_store(a.whead, a.nbp, d, pf));
    }
    phase_store(a, a.whead, a.nbp, d, hpr, hlo, logr, a.nbp, j, sm, pf);
  }
  AMS_SYNC((void)0);
#undef AMS_SYNC
  if (blockIdx.x == 0) phase_feed(a, a.A - 1, false, sm);
  return;
failed:
  // a barrier that timed out: the step's tokens all read -1 (workgroup 0 owns them)
  // and the host-visible status word reports it to the next call on the context
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < M * a.A; i += blockDim.x) a.out_tok[i] = -1;
  if (threadIdx.x == 0 && a.status) __hip_atomic_store(a.status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ void k_fused_reset(unsigned* sync, int words) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < words; i += gridDim.x * blockDim.x) sync[i] = 0u;
}

int fused_sync_words(int d, int H) { return SYNC_STRIP + (d / 16 > 8 * H ? d / 16 : 8 * H); }

// Largest grid that is resident at once: one workgroup per compute unit when
// the kernel fits (0 if not).
int decode_fused_grid(int device, int dh) {
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return 0;
  const hipError_t e = dh == 64
                           ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_decode_fused<64>, 512, 0)
                           : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_decode_fused<128>, 512, 0);
  if (e != hipSuccess || per_cu < 1) return 0;
  return cus;
}

hipError_t decode_fused(const FusedDecode& f, int grid, hipStream_t s) {
  FusedArgs a;
  a.wqkv = (const f16*)f.wqkv; a.s_qkv = f.s_qkv;
  a.wo = (const f16*)f.wo; a.s_o = f.s_o;
  a.wgu = (const f16*)f.wgu; a.s_gu = f.s_gu;
  a.wd = (const f16*)f.wd; a.s_d = f.s_d;
  a.whead = (const f16*)f.whead;
  a.bin_embed = (const f16*)f.bin_embed;
  a.L = f.L; a.d = f.d; a.H = f.H; a.F = f.F; a.nbp = f.nbp; a.n_bins = f.n_bins;
  a.eps = f.eps;
  a.scale = 1.0f / sqrtf((float)f.dh);
  a.M = f.M; a.cap = f.cap; a.A = f.A;
  a.split_o = f.split_o; a.split_d = f.split_d; a.split_a = f.split_a;
  a.lens = f.lens; a.rope = f.rope;
  a.kv = (f16*)f.kv; a.slab = f.slab_elems;
  a.pt = f.pt; a.ppr = f.ppr;
  a.h = f.h; a.hp = (f16*)f.hp;
  a.hl = (const f16*)f.hl; a.hl_lo = (uint32_t)((const char*)f.hl_lo - (const char*)f.hl);
  a.qkv = f.qkv; a.op = (f16*)f.op; a.ap = (f16*)f.ap;
  a.logits = f.logits; a.part = f.part; a.sync = f.sync; a.status = f.status;
  a.out_tok = f.out_tok; a.out_logits = f.out_logits; a.forced = f.forced;
  const int words = fused_sync_words(f.d, f.H);
  hipLaunchKernelGGL(k_fused_reset, dim3((words + 255) / 256), dim3(256), 0, s, f.sync, words);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (f.dh == 64) hipLaunchKernelGGL(k_decode_fused<64>, dim3(grid), dim3(512), 0, s, a);
  else hipLaunchKernelGGL(k_decode_fused<128>, dim3(grid), dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace ams

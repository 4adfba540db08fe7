// Two-phase hashing for the action index (paper section 3.2.3, "Virtual Action",
// Algorithm 1 "Two-Phase Hashing for Action Index") and the page keys of
// prefixes built on it.
//
// Phase 1 hashes every s-byte segment of the input on its own, phase 2 merges
// the segment hashes in order.  Both hash functions are polynomial hashes
// modulo the Mersenne prime 2^31 - 1, evaluated with two independent bases
// whose 31-bit results are packed into one 64-bit value (first base low):
//   HashFunc1(B_i) = (sum_j u_j r^(s/2-1-j)) r + |B_i|, u_j the 16-bit
//                    little-endian units of B_i zero-padded to s bytes;
//   HashFunc2(h_1..h_k) = (sum_i h_i q^(k-i)) q + N.
//
// Phase 1: one workgroup of 256 threads per segment.  Each thread evaluates
// the polynomial of 8 consecutive units (one 16-byte load) and the 256 pieces
// are combined pairwise in order (left * base^len(right) + right) through wave
// shuffles and LDS; a segment of fewer than 2048 units is right-aligned so
// that the idle leading threads contribute the polynomial's leading zeros, and
// longer segments go block by block.  The work is integer ALU on data read once
// from HBM.
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace ams {

namespace {

constexpr uint64_t M31 = 0x7FFFFFFFull;
constexpr uint32_t HR0 = 0x2545F491u, HR1 = 0x1B873593u;  // HashFunc1 bases
constexpr uint32_t HQ0 = 0x3C6EF372u, HQ1 = 0x0A54FF53u;  // HashFunc2 bases

__device__ __forceinline__ uint64_t red(uint64_t x) {  // x < 2^63 -> x mod (2^31 - 1)
  x = (x & M31) + (x >> 31);
  x = (x & M31) + (x >> 31);
  return x >= M31 ? x - M31 : x;
}
__device__ __forceinline__ uint64_t mulm(uint64_t a, uint64_t b) { return red(a * b); }  // a, b < 2^31
__device__ __forceinline__ uint64_t addm(uint64_t a, uint64_t b) { return red(a + b); }
__device__ uint64_t powm(uint64_t b, uint64_t e) {
  uint64_t r = 1;
  while (e) {
    if (e & 1) r = mulm(r, b);
    b = mulm(b, b);
    e >>= 1;
  }
  return r;
}

// In-order combination of the 256 threads' (value, piece) pairs of one block:
// value(left ++ right) = value(left) * base^len(right) + value(right); at level l
// every piece spans 8 * 2^l units.  pw[l] = base^(8 * 2^l).  Returns the
// block's value in thread 0.
__device__ uint64_t tree256(uint64_t v, const uint64_t* pw, uint64_t* lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int l = 0; l < 6; ++l) {
    const int w = 1 << l;
    const uint64_t right = (uint64_t)__shfl_down((unsigned long long)v, w, 64);
    if ((lane & (2 * w - 1)) == 0) v = addm(mulm(v, pw[l]), right);
  }
  if (lane == 0) lds[wave] = v;
  __syncthreads();
  uint64_t out = 0;
  if (threadIdx.x == 0) {
    const uint64_t a = addm(mulm(lds[0], pw[6]), lds[1]);
    const uint64_t b = addm(mulm(lds[2], pw[6]), lds[3]);
    out = addm(mulm(a, pw[7]), b);
  }
  __syncthreads();
  return out;
}

__device__ __forceinline__ uint64_t horner8(const uint32_t (&w)[4], uint64_t base) {
  uint64_t v = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v = addm(mulm(v, base), w[i] & 0xFFFFu);
    v = addm(mulm(v, base), w[i] >> 16);
  }
  return v;
}

// Phase 1.  Segment g = blockIdx.x covers bytes [g s, g s + s) of data (zero
// beyond n_bytes).  s is a multiple of 16 and data is 16-byte aligned.
__global__ __launch_bounds__(256) void k_hash_segments(const uint8_t* __restrict__ data, uint64_t n_bytes, int s,
                                                       uint64_t* __restrict__ seg_out) {
  __shared__ uint64_t lds[2][4];
  __shared__ uint64_t pws[2][8];
  const uint64_t g = blockIdx.x;
  const uint64_t base = g * (uint64_t)s;
  const int U = s / 2, nblk = (U + 2047) / 2048;
  if (threadIdx.x < 2) {
    const uint64_t r = threadIdx.x == 0 ? HR0 : HR1;
    uint64_t p = powm(r, 8);
    for (int l = 0; l < 8; ++l) {
      pws[threadIdx.x][l] = p;
      p = mulm(p, p);
    }
  }
  __syncthreads();
  uint64_t acc0 = 0, acc1 = 0;  // thread 0: the segment's value so far
  for (int b = 0; b < nblk; ++b) {
    const int units = min(2048, U - b * 2048);  // a multiple of 8
    const int chunks = units / 8;
    const int c = (int)threadIdx.x - (256 - chunks);  // right-aligned
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (c >= 0) {
      const uint64_t off = base + 2ull * (b * 2048 + 8 * c);  // byte offset of the thread's 16 bytes
      if (off + 16 <= n_bytes) {
        const uint4 q = *reinterpret_cast<const uint4*>(data + off);
        w[0] = q.x; w[1] = q.y; w[2] = q.z; w[3] = q.w;
      } else if (off < n_bytes) {
        for (uint64_t i = off; i < n_bytes; ++i) w[(i - off) >> 2] |= (uint32_t)data[i] << (8 * ((i - off) & 3));
      }
    }
    const uint64_t v0 = tree256(horner8(w, HR0), pws[0], lds[0]);
    const uint64_t v1 = tree256(horner8(w, HR1), pws[1], lds[1]);
    if (threadIdx.x == 0) {  // Horner over blocks: acc r^units + block
      acc0 = addm(mulm(acc0, powm(HR0, units)), v0);
      acc1 = addm(mulm(acc1, powm(HR1, units)), v1);
    }
  }
  if (threadIdx.x == 0) {
    const uint64_t len = n_bytes - base < (uint64_t)s ? n_bytes - base : (uint64_t)s;
    const uint64_t h0 = addm(mulm(acc0, HR0), red(len));
    const uint64_t h1 = addm(mulm(acc1, HR1), red(len));
    seg_out[g] = h0 | (h1 << 32);
  }
}

// Phase 2 over k segment hashes: 256 threads, thread t merging the virtual
// range [t m, t m + m) of a right-aligned index space (m = ceil(k / 256)), then
// the in-order tree with q^(m 2^l).  out = (value) q + n_bytes per component.
__global__ __launch_bounds__(256) void k_hash_merge(const uint64_t* __restrict__ seg, uint64_t k, uint64_t n_bytes,
                                                    uint64_t* __restrict__ out) {
  __shared__ uint64_t lds[2][4];
  __shared__ uint64_t pws[2][8];
  const uint64_t m = (k + 255) / 256, lead = 256 * m - k;
  if (threadIdx.x < 2) {
    const uint64_t q = threadIdx.x == 0 ? HQ0 : HQ1;
    uint64_t p = powm(q, m);
    for (int l = 0; l < 8; ++l) {
      pws[threadIdx.x][l] = p;
      p = mulm(p, p);
    }
  }
  __syncthreads();
  uint64_t v0 = 0, v1 = 0;
  for (uint64_t j = 0; j < m; ++j) {
    const uint64_t vi = threadIdx.x * m + j;
    const uint64_t h = vi >= lead ? seg[vi - lead] : 0ull;
    v0 = addm(mulm(v0, HQ0), h & 0xFFFFFFFFull);
    v1 = addm(mulm(v1, HQ1), h >> 32);
  }
  // tree256 assumes pieces of 8 * 2^l units; here a piece at level l spans m 2^l
  // segments, which pws already encodes (pws[l] = q^(m 2^l))
  const uint64_t t0 = tree256(v0, pws[0], lds[0]);
  const uint64_t t1 = tree256(v1, pws[1], lds[1]);
  if (threadIdx.x == 0) {
    const uint64_t H0 = addm(mulm(t0, HQ0), red(n_bytes % M31));
    const uint64_t H1 = addm(mulm(t1, HQ1), red(n_bytes % M31));
    out[0] = H0 | (H1 << 32);
  }
}

// Page keys of packed rows: row b spans row_bytes[b] bytes whose segment
// hashes (the row's bytes start on a segment boundary) sit from seg +
// seg_first[b] on.  Key of page m (m < floor(row_bytes / page_bytes)) =
// HashFunc2 of the row's segments covering its first (m + 1) page_bytes bytes.
// One thread per row (a sequential scan of a few hundred segments).
__global__ void k_hash_page_keys(const uint64_t* __restrict__ seg, const int64_t* __restrict__ seg_first,
                                 const int64_t* __restrict__ row_bytes, int B, int64_t page_bytes, int s,
                                 int max_pages, uint64_t* __restrict__ keys) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int64_t per_page = page_bytes / s, n_pages = min<int64_t>(row_bytes[b] / page_bytes, max_pages);
  const uint64_t* sg = seg + seg_first[b];
  uint64_t a0 = 0, a1 = 0;
  for (int64_t pg = 0; pg < n_pages; ++pg) {
    for (int64_t i = pg * per_page; i < (pg + 1) * per_page; ++i) {
      a0 = addm(mulm(a0, HQ0), sg[i] & 0xFFFFFFFFull);
      a1 = addm(mulm(a1, HQ1), sg[i] >> 32);
    }
    const uint64_t len = red((uint64_t)((pg + 1) * page_bytes) % M31);
    keys[(size_t)b * max_pages + pg] = addm(mulm(a0, HQ0), len) | (addm(mulm(a1, HQ1), len) << 32);
  }
}

}  // namespace

// Scratch of the allocation-free index hash (ams_index_hash_noalloc): the
// phase-1 segment hashes of one call, at most INDEX_NOALLOC_MAX_SEGMENTS of
// them (1 MiB).  Every device the library runs on holds its own copy until the
// process ends, and every call on that device shares it.  Host code never
// passes the array's name to a kernel: it takes the device address that
// hipGetSymbolAddress returned for the current device (index_noalloc_scratch).
static __device__ __align__(256) uint64_t scratch[INDEX_NOALLOC_MAX_SEGMENTS];

namespace {
std::mutex g_scratch_mu;
uint64_t* g_scratch_ptr[64] = {};  // per device id
}  // namespace

hipError_t index_noalloc_scratch(int device, uint64_t** ptr) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (device < 0 || device >= 64) return hipErrorInvalidDevice;
  if (!g_scratch_ptr[device]) {  // once per device, with that device current
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = (uint64_t*)p;
  }
  *ptr = g_scratch_ptr[device];
  return hipSuccess;
}

hipError_t hash_segments(const void* data, uint64_t n_bytes, int s, uint64_t* seg_out, hipStream_t st) {
  const uint64_t k = (n_bytes + s - 1) / s;
  if (k == 0) return hipSuccess;
  hipLaunchKernelGGL(k_hash_segments, dim3((unsigned)k), dim3(256), 0, st, (const uint8_t*)data, n_bytes, s, seg_out);
  return hipGetLastError();
}

hipError_t hash_merge(const uint64_t* seg, uint64_t k, uint64_t n_bytes, uint64_t* out, hipStream_t st) {
  hipLaunchKernelGGL(k_hash_merge, dim3(1), dim3(256), 0, st, seg, k, n_bytes, out);
  return hipGetLastError();
}

hipError_t hash_page_keys(const uint64_t* seg, const int64_t* seg_first, const int64_t* row_bytes, int B,
                          int64_t page_bytes, int s, int max_pages, uint64_t* keys, hipStream_t st) {
  hipLaunchKernelGGL(k_hash_page_keys, dim3((B + 63) / 64), dim3(64), 0, st, seg, seg_first, row_bytes, B,
                     page_bytes, s, max_pages, keys);
  return hipGetLastError();
}

}  // namespace ams

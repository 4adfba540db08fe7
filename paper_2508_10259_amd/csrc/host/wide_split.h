// The balanced split of the wide decode GEMM, shared by the kernel and the
// host-side planning (plain C++: the host bookkeeping also builds without HIP;
// constexpr functions are callable from device code).
//
// The (128-row weight tile, 128-wide K chunk) units of an N x K projection,
// tile by tile (U = N/128 * K/128 of them), are cut into P contiguous shares:
// workgroup w takes units [floor(w U / P), floor((w+1) U / P)).  P <= U, so
// every share holds a unit and the workgroups of a tile are consecutive.
#pragma once

namespace ams {

// The workgroup holding unit a: the largest w with floor(w U / P) <= a.
constexpr int wide_unit_owner(long long a, int P, long long U) { return (int)(((a + 1) * P - 1) / U); }

// Workgroups of the balanced split: `wgs`, at most one per unit.
inline int wide_stream_wgs(int N, int K, int wgs) {
  const long long U = (long long)(N / 128) * (K / 128);
  return (int)(wgs < U ? wgs : U);
}

// Partial-sum slots of the balanced split: the most workgroups any tile meets.
inline int wide_stream_slots(int N, int K, int wgs) {
  const int nch = K / 128, T = N / 128;
  const long long U = (long long)T * nch;
  const int P = wide_stream_wgs(N, K, wgs);
  int best = 1;
  for (int t = 0; t < T; ++t) {
    const int c = wide_unit_owner((long long)(t + 1) * nch - 1, P, U) - wide_unit_owner((long long)t * nch, P, U) + 1;
    best = c > best ? c : best;
  }
  return best;
}

}  // namespace ams

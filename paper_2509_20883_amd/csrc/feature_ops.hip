// Feature transforms fused over many columns (gfx950): bucketize and mod
// (RecIS, "Bucketize and Mod" among the benchmarked operators: a model holds
// dozens to hundreds of them, and one launch for all columns replaces one
// launch per column).
//
// Column c holds elements [col_off[c], col_off[c+1]) of one flat array.  A
// block takes 1024 consecutive elements and copies the column offsets (and
// the boundary offsets or moduli) to LDS in one coalesced trip; it finds the
// columns its range spans there.  When the range lies inside one column (the
// usual case: columns are much longer than a block) it stages that column's
// boundaries in LDS and every element searches there; otherwise each element
// searches its column, then the boundaries in global memory (L1 / L2).
//   bucketize: out = number of boundaries b <= x (upper bound)
//   mod:       out = x mod m in [0, m) (-1 for a modulus <= 0)
#include "device_common.h"

namespace rs {

constexpr int kFeatItems = 4;
constexpr int kFeatTile = kBlock * kFeatItems;  // 1024 elements per block
constexpr int kLdsBounds = 4096;               // boundaries staged in LDS

// Largest c in [lo, hi] with off[c] <= i (off nondecreasing, off[lo] <= i).
template <typename P>
__device__ inline int column_of(P off, int lo, int hi, int64_t i) {
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Upper bound: the index of the first of b[0, nb) (nondecreasing) with
// x < b, or nb -- the number of boundaries b <= x, and nb for a NaN x (which
// compares below no boundary).
template <typename P>
__device__ inline int64_t upper_bound_f(P b, int64_t nb, float x) {
  int64_t lo = 0, hi = nb;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (x < b[mid]) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

// Up to kLdsCols column offsets (and one per-column array: boundary offsets
// or moduli) are copied to LDS in one coalesced trip, so the column searches
// run in LDS; with more columns they run in global memory (L1 / L2).
constexpr int kLdsCols = 1024;

template <typename T>
__device__ inline void stage_columns(const int64_t* __restrict__ col_off, const T* __restrict__ aux, int naux,
                                     int ncols, int64_t* lco, T* laux) {
  for (int c = threadIdx.x; c <= ncols; c += kBlock) lco[c] = col_off[c];
  for (int c = threadIdx.x; c < naux; c += kBlock) laux[c] = aux[c];
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void k_bucketize(const float* __restrict__ values, int64_t n,
                                                      const int64_t* __restrict__ col_off, int ncols,
                                                      const float* __restrict__ bnd,
                                                      const int64_t* __restrict__ bnd_off, int64_t* __restrict__ out) {
  __shared__ float lb[kLdsBounds];
  __shared__ int64_t lco[kLdsCols];
  __shared__ int64_t lbo[kLdsCols];
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * kFeatTile;
  const int64_t b1 = min(b0 + kFeatTile, n);
  float x[kFeatItems];
#pragma unroll
  for (int k = 0; k < kFeatItems; ++k) {  // in flight while the offsets are staged
    const int64_t i = b0 + k * kBlock + threadIdx.x;
    x[k] = i < b1 ? values[i] : 0.0f;
  }
  const bool lds = ncols < kLdsCols;  // ncols + 1 offsets fit
  if (lds) stage_columns(col_off, bnd_off, ncols + 1, ncols, lco, lbo);
  const int c0 = lds ? column_of(static_cast<const int64_t*>(lco), 0, ncols - 1, b0)
                     : column_of(col_off, 0, ncols - 1, b0);
  const int c1 = lds ? column_of(static_cast<const int64_t*>(lco), c0, ncols - 1, b1 - 1)
                     : column_of(col_off, c0, ncols - 1, b1 - 1);
  if (c0 == c1) {  // block-uniform
    const int64_t o = lds ? lbo[c0] : bnd_off[c0];
    const int64_t nb = (lds ? lbo[c0 + 1] : bnd_off[c0 + 1]) - o;
    if (nb <= kLdsBounds) {
      for (int64_t j = threadIdx.x; j < nb; j += kBlock) lb[j] = bnd[o + j];
      __syncthreads();
#pragma unroll
      for (int k = 0; k < kFeatItems; ++k) {
        const int64_t i = b0 + k * kBlock + threadIdx.x;
        if (i < b1) out[i] = upper_bound_f(static_cast<const float*>(lb), nb, x[k]);
      }
      return;
    }
  }
#pragma unroll
  for (int k = 0; k < kFeatItems; ++k) {
    const int64_t i = b0 + k * kBlock + threadIdx.x;
    if (i >= b1) continue;
    const int c = lds ? column_of(static_cast<const int64_t*>(lco), c0, c1, i) : column_of(col_off, c0, c1, i);
    const int64_t o = lds ? lbo[c] : bnd_off[c];
    const int64_t e = lds ? lbo[c + 1] : bnd_off[c + 1];
    out[i] = upper_bound_f(bnd + o, e - o, x[k]);
  }
}

__device__ inline int64_t floor_mod(int64_t x, int64_t m) {
  const int64_t r = x % m;
  return r < 0 ? r + m : r;
}

__global__ __launch_bounds__(kBlock) void k_mod(const int64_t* __restrict__ values, int64_t n,
                                                const int64_t* __restrict__ col_off, int ncols,
                                                const int64_t* __restrict__ moduli, int64_t* __restrict__ out) {
  __shared__ int64_t lco[kLdsCols];
  __shared__ int64_t lm[kLdsCols];
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * kFeatTile;
  const int64_t b1 = min(b0 + kFeatTile, n);
  int64_t x[kFeatItems];
#pragma unroll
  for (int k = 0; k < kFeatItems; ++k) {
    const int64_t i = b0 + k * kBlock + threadIdx.x;
    x[k] = i < b1 ? values[i] : 0;
  }
  const bool lds = ncols < kLdsCols;
  if (lds) stage_columns(col_off, moduli, ncols, ncols, lco, lm);
  const int c0 = lds ? column_of(static_cast<const int64_t*>(lco), 0, ncols - 1, b0)
                     : column_of(col_off, 0, ncols - 1, b0);
  const int c1 = lds ? column_of(static_cast<const int64_t*>(lco), c0, ncols - 1, b1 - 1)
                     : column_of(col_off, c0, ncols - 1, b1 - 1);
  const int64_t m0 = lds ? lm[c0] : moduli[c0];
#pragma unroll
  for (int k = 0; k < kFeatItems; ++k) {
    const int64_t i = b0 + k * kBlock + threadIdx.x;
    if (i >= b1) continue;
    int64_t m = m0;
    if (c0 != c1) {
      const int c = lds ? column_of(static_cast<const int64_t*>(lco), c0, c1, i) : column_of(col_off, c0, c1, i);
      m = lds ? lm[c] : moduli[c];
    }
    const int64_t r = floor_mod(x[k], m > 0 ? m : 1);
    out[i] = m > 0 ? r : -1;  // a modulus <= 0 is no bucket
  }
}

hipError_t launch_bucketize(const float* values, int64_t n, const int64_t* col_off, int ncols, const float* bnd,
                            const int64_t* bnd_off, int64_t* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_bucketize<<<grid_for(n, kFeatTile, 1ll << 31), kBlock, 0, s>>>(values, n, col_off, ncols, bnd, bnd_off, out);
  return hipGetLastError();
}

hipError_t launch_mod(const int64_t* values, int64_t n, const int64_t* col_off, int ncols, const int64_t* moduli,
                      int64_t* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_mod<<<grid_for(n, kFeatTile, 1ll << 31), kBlock, 0, s>>>(values, n, col_off, ncols, moduli, out);
  return hipGetLastError();
}

}  // namespace rs

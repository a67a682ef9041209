// Bandwidth probes (gfx950): plain device operations that bound what the
// embedding step's kernels can reach on this GPU, measured with the same
// access widths and launch shapes (16-byte lane accesses, 256-thread blocks,
// lane groups of up to 64 lanes per row, each lane moving 16-byte words).  They are measurement
// references only; no step uses them.
//   kProbeRead    sequential read of `bytes` (every 16-byte word summed)
//   kProbeWrite   sequential streaming write of `bytes` (non-temporal stores)
//   kProbeCopy    sequential copy of `bytes` (read + non-temporal write)
//   kProbeGather  out[i] = rows[idx[i]] for n rows of row_bytes: random row
//                 reads, one streamed output row per index
//   kProbeRmw     rows[idx[i]] += 1 for n rows of row_bytes: random row
//                 read-modify-write in place (as the optimizer does, the
//                 write non-temporal)
#include "device_common.h"

#include <hip/hip_ext.h>

namespace rs {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// The streaming probes make one pass: thread t of block b moves 16-byte word
// b * 256 + t, so the blocks, dispatched in order, sweep the buffer once
// (measured on this GPU: a grid-stride loop over 2048-8192 blocks writes at
// 4.4-5.2 TB/s, one pass at 6.9-7.1 TB/s).

__global__ __launch_bounds__(kBlock) void k_probe_read(const uint4* __restrict__ a, int64_t n16,
                                                       uint32_t* __restrict__ sink) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n16) return;
  const uint4 v = a[i];
  // a store the compiler cannot drop; taken only for one specific word
  if ((v.x ^ v.y ^ v.z ^ v.w) == 0x9E3779B9u) sink[0] = v.x;
}

__global__ __launch_bounds__(kBlock) void k_probe_write(uint4* __restrict__ a, int64_t n16, uint32_t value) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n16) return;
  const u32x4 v = {value, value, value, value};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(a + i));
}

__global__ __launch_bounds__(kBlock) void k_probe_copy(const uint4* __restrict__ a, uint4* __restrict__ b,
                                                       int64_t n16) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n16) return;
  const uint4 v = a[i];
  const u32x4 x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(b + i));
}

// Lane groups of `lanes` lanes, each lane moving nch 16-byte words of a row
// (at lane * 16 + c * lanes * 16), kRows rows in flight per group.  Indices
// outside [0, nrows) are skipped (their output row is not written).
constexpr int kProbeMaxChunks = 4;

template <int kRows>
__global__ __launch_bounds__(kBlock) void k_probe_gather(const uint8_t* __restrict__ rows, int64_t nrows, int row_bytes,
                                                         int lanes, int nch, const int64_t* __restrict__ idx,
                                                         int64_t n, uint8_t* __restrict__ out) {
  const int lane = threadIdx.x % lanes, grp = threadIdx.x / lanes, gpb = kBlock / lanes;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * gpb * kRows;
  for (int64_t i0 = (static_cast<int64_t>(blockIdx.x) * gpb + grp) * kRows; i0 < n; i0 += stride) {
    int64_t r[kRows];
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      r[k] = i0 + k < n ? idx[i0 + k] : -1;
      if (r[k] >= nrows) r[k] = -1;
    }
    uint4 v[kRows][kProbeMaxChunks];
#pragma unroll
    for (int k = 0; k < kRows; ++k)
#pragma unroll
      for (int c = 0; c < kProbeMaxChunks; ++c)
        v[k][c] = r[k] >= 0 && c < nch
                      ? *reinterpret_cast<const uint4*>(rows + r[k] * row_bytes + (c * lanes + lane) * 16)
                      : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      if (r[k] < 0) continue;
#pragma unroll
      for (int c = 0; c < kProbeMaxChunks; ++c) {
        if (c >= nch) continue;
        const u32x4 x = {v[k][c].x, v[k][c].y, v[k][c].z, v[k][c].w};
        __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(out + (i0 + k) * row_bytes + (c * lanes + lane) * 16));
      }
    }
  }
}

template <int kRows>
__global__ __launch_bounds__(kBlock) void k_probe_rmw(uint8_t* __restrict__ rows, int64_t nrows, int row_bytes, int lanes,
                                                      int nch, const int64_t* __restrict__ idx, int64_t n) {
  const int lane = threadIdx.x % lanes, grp = threadIdx.x / lanes, gpb = kBlock / lanes;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * gpb * kRows;
  for (int64_t i0 = (static_cast<int64_t>(blockIdx.x) * gpb + grp) * kRows; i0 < n; i0 += stride) {
    int64_t r[kRows];
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      r[k] = i0 + k < n ? idx[i0 + k] : -1;
      if (r[k] >= nrows) r[k] = -1;
    }
    float4 v[kRows][kProbeMaxChunks];
#pragma unroll
    for (int k = 0; k < kRows; ++k)
#pragma unroll
      for (int c = 0; c < kProbeMaxChunks; ++c)
        if (r[k] >= 0 && c < nch)
          v[k][c] = *reinterpret_cast<const float4*>(rows + r[k] * row_bytes + (c * lanes + lane) * 16);
#pragma unroll
    for (int k = 0; k < kRows; ++k) {
      if (r[k] < 0) continue;
#pragma unroll
      for (int c = 0; c < kProbeMaxChunks; ++c) {
        if (c >= nch) continue;
        // written back non-temporally, as the optimizer's update is
        const nt_f32x4 x = {v[k][c].x + 1.f, v[k][c].y + 1.f, v[k][c].z + 1.f, v[k][c].w + 1.f};
        __builtin_nontemporal_store(x, reinterpret_cast<nt_f32x4*>(rows + r[k] * row_bytes + (c * lanes + lane) * 16));
      }
    }
  }
}

// Lanes per row for a row of w16 16-byte words: the largest power of two
// <= 64 dividing w16 that leaves at most kProbeMaxChunks words per lane, or 0.
int probe_lanes(int w16) {
  for (int l = 64; l >= 1; l >>= 1)
    if (w16 % l == 0) return w16 / l <= kProbeMaxChunks ? l : 0;
  return 0;
}

hipError_t launch_probe(int kind, void* a, int64_t a_bytes, void* b, const int64_t* idx, int64_t n, int row_bytes,
                        hipStream_t s) {
  switch (kind) {
    case kProbeRead:
      k_probe_read<<<grid_for(n / 16, kBlock, int64_t(1) << 31), kBlock, 0, s>>>(static_cast<const uint4*>(a), n / 16,
                                                                                static_cast<uint32_t*>(b));
      break;
    case kProbeWrite:
      k_probe_write<<<grid_for(n / 16, kBlock, int64_t(1) << 31), kBlock, 0, s>>>(static_cast<uint4*>(a), n / 16,
                                                                                 0x3F800000u);
      break;
    case kProbeCopy:
      k_probe_copy<<<grid_for(n / 16, kBlock, int64_t(1) << 31), kBlock, 0, s>>>(static_cast<const uint4*>(a),
                                                                                static_cast<uint4*>(b), n / 16);
      break;
    case kProbeGather:
    case kProbeRmw: {
      constexpr int kRows = 8;
      const int lanes = row_bytes % 16 == 0 ? probe_lanes(row_bytes / 16) : 0;
      if (lanes == 0) return hipErrorInvalidValue;
      const int nch = row_bytes / 16 / lanes;
      const unsigned g = grid_for(n, static_cast<int64_t>(kBlock / lanes) * kRows, int64_t(1) << 31);  // one pass
      if (kind == kProbeGather)
        k_probe_gather<kRows><<<g, kBlock, 0, s>>>(static_cast<const uint8_t*>(a), a_bytes / row_bytes, row_bytes,
                                                   lanes, nch, idx, n, static_cast<uint8_t*>(b));
      else
        k_probe_rmw<kRows><<<g, kBlock, 0, s>>>(static_cast<uint8_t*>(a), a_bytes / row_bytes, row_bytes, lanes, nch,
                                                idx, n);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rs

// Channels-last pooling of one (image, channel block) by a workgroup of
// kPoolThreads threads (Sec. 3.3: the descriptor is the spatial mean of each
// channel); 512 threads, so that several workgroups share a CU and small
// images still keep enough loads in flight.  Lane l of the 32-lane row groups
// reads the 16-byte channel vector l of the block; row group r takes
// positions r, r + kPoolGroups, ..., four of them per round with all four
// loads in flight.  The kPoolGroups partial sums of each channel are then
// added in a fixed order through LDS, so the result does not depend on
// timing.
#pragma once

#include "moce_internal.h"

namespace moce {

constexpr int kPoolThreads = 512;
constexpr int kPoolGroups = kPoolThreads / 32;  // row groups

template <typename T> struct PoolVec;
template <> struct PoolVec<uint16_t> {
  static constexpr int EPV = 8;
  __device__ static void add(const uint4& v, float (&a)[8]) {
    a[0] += bf16_lo(v.x); a[1] += bf16_hi(v.x); a[2] += bf16_lo(v.y); a[3] += bf16_hi(v.y);
    a[4] += bf16_lo(v.z); a[5] += bf16_hi(v.z); a[6] += bf16_lo(v.w); a[7] += bf16_hi(v.w);
  }
};
template <> struct PoolVec<float> {
  static constexpr int EPV = 4;
  __device__ static void add(const uint4& v, float (&a)[4]) {
    a[0] += __uint_as_float(v.x); a[1] += __uint_as_float(v.y);
    a[2] += __uint_as_float(v.z); a[3] += __uint_as_float(v.w);
  }
};

// Channels of block cb: 32 EPV of them from channel 32 EPV cb (C a multiple of
// EPV).  A block with nv < 32 vectors (C below 32 EPV) gives each vector
// rep = 32 / nv lanes of a row group, which take positions in turn, so that
// no lane idles; with nv = 32 lane l reads vector l at positions rg,
// rg + 32, ...  `part` is LDS of kPoolGroups * 32 * EPV floats.  The mean of
// channel c of image b goes to d[b sb + c sc]: sb = C, sc = 1 for d[B][C],
// sb = 1, sc = B for its transpose.
template <typename T>
__device__ __forceinline__ void pool_rows_block(const T* __restrict__ x, float* __restrict__ d, int C, int HW,
                                                int64_t b, int cb, float* part, int64_t sb, int64_t sc) {
  constexpr int EPV = PoolVec<T>::EPV;
  const int l = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const int nv = min(32, C / EPV - 32 * cb);
  const int rep = 32 / nv;
  const int v = l % nv, sub = l / nv;
  const int c0 = (cb * 32 + v) * EPV;
  float acc[EPV];
#pragma unroll
  for (int j = 0; j < EPV; ++j) acc[j] = 0.f;
  if (sub < rep) {
    const T* col = x + b * HW * (int64_t)C + c0;
    const int stride = kPoolGroups * rep;  // positions between a lane's consecutive reads
    for (int p0 = rg * rep + sub; p0 < HW; p0 += 4 * stride) {
      uint4 vv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int p = min(p0 + u * stride, HW - 1);
        vv[u] = *reinterpret_cast<const uint4*>(col + (int64_t)p * C);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (p0 + u * stride < HW) PoolVec<T>::add(vv[u], acc);
    }
  }
#pragma unroll
  for (int j = 0; j < EPV; ++j) part[(rg * 32 + l) * EPV + j] = acc[j];
  __syncthreads();
  // channel i of the block: the partial sums of its rep lanes in each of the
  // 32 row groups, in a fixed order
  for (int i = threadIdx.x; i < nv * EPV; i += kPoolThreads) {
    const int vi = i / EPV, j = i - vi * EPV;
    float s = 0.f;
    for (int r = 0; r < kPoolGroups; ++r)
      for (int m = 0; m < rep; ++m) s += part[(r * 32 + vi + m * nv) * EPV + j];
    d[b * sb + (int64_t)(cb * 32 * EPV + i) * sc] = s / (float)HW;
  }
}

}  // namespace moce

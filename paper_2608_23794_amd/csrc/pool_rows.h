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

// Channels-first bfloat16 planes of H W positions, H W a multiple of 4 (so
// every plane starts 8-byte aligned): L lanes per plane read 8-byte pieces,
// four per lane in flight.  Lane group `group` of `ngroups` takes planes
// group, group + ngroups, ...; a plane's sum depends only on L, so every
// launch shape with the same L gives the same bits.
inline int planes8_lanes(int64_t HW) {
  const int64_t nq = HW / 4;
  return nq >= 192 ? 64 : nq >= 96 ? 32 : nq >= 32 ? 16 : 8;
}

template <int L>
__device__ __forceinline__ void pool_planes8(const uint16_t* __restrict__ x, float* __restrict__ d, int64_t planes,
                                             int HW, int64_t group, int64_t ngroups) {
  const int lane = threadIdx.x % L;
  const int nq = HW / 4;
  for (int64_t pl = group; pl < planes; pl += ngroups) {
    const uint2* q = reinterpret_cast<const uint2*>(x + pl * HW);
    float sum = 0.f;
    for (int v0 = lane; v0 < nq; v0 += 4 * L) {
      uint2 buf[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) buf[u] = q[min(v0 + u * L, nq - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (v0 + u * L < nq) sum += (bf16_lo(buf[u].x) + bf16_hi(buf[u].x)) + (bf16_lo(buf[u].y) + bf16_hi(buf[u].y));
    }
    sum = wave_sum<L>(sum);
    if (lane == 0) d[pl] = sum / (float)HW;
  }
}

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

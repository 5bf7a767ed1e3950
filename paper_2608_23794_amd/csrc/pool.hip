// Global average pooling descriptor z = GAP(x) (Sec. 3.3).
//
// NCHW: a group of L lanes (L = 8..64, chosen from the plane length) reduces
// one H*W plane with 16-byte loads.  A plane's start is 16-byte aligned only
// when H*W*elem is a multiple of 16, so each plane is read as an unaligned
// head, an aligned vector body and a tail; every byte of x is read once.
// NHWC: lanes map to 16-byte channel vectors of a position row (consecutive
// lanes read consecutive bytes), the four waves of a block split the rows,
// and the four partial sums meet in LDS.
#include <algorithm>

#include "moce_internal.h"
#include "pool_rows.h"

namespace moce {
namespace {

template <typename T> __device__ __forceinline__ float load_elem(const T* p);
template <> __device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

template <typename T> __device__ __forceinline__ float sum16(uint4 v);
template <> __device__ __forceinline__ float sum16<float>(uint4 v) {
  return (__uint_as_float(v.x) + __uint_as_float(v.y)) + (__uint_as_float(v.z) + __uint_as_float(v.w));
}
template <> __device__ __forceinline__ float sum16<uint16_t>(uint4 v) {
  return ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
         ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
}

template <typename T, int L>
__global__ void __launch_bounds__(256)
k_pool_nchw(const T* __restrict__ x, float* __restrict__ d, int64_t planes, int HW) {
  constexpr int EPV = 16 / sizeof(T);  // elements per 16-byte vector
  const int lane = threadIdx.x % L;
  const int64_t group = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / L;
  const int64_t ngroups = ((int64_t)gridDim.x * blockDim.x) / L;
  for (int64_t pl = group; pl < planes; pl += ngroups) {
    const T* base = x + pl * HW;
    const uintptr_t addr = reinterpret_cast<uintptr_t>(base);
    int head = (int)(((16u - (addr & 15u)) & 15u) / sizeof(T));
    if (head > HW) head = HW;
    const int nvec = (HW - head) / EPV;
    const int tail0 = head + nvec * EPV;
    float sum = 0.f;
    for (int e = lane; e < head; e += L) sum += load_elem<T>(base + e);
    const uint4* vb = reinterpret_cast<const uint4*>(base + head);
    for (int v = lane; v < nvec; v += L) sum += sum16<T>(vb[v]);
    for (int e = tail0 + lane; e < HW; e += L) sum += load_elem<T>(base + e);
    sum = wave_sum<L>(sum);
    if (lane == 0) d[pl] = sum / (float)HW;
  }
}

// Planes whose length is a whole number of 16-byte vectors (so every plane
// starts 16-byte aligned): one wave per plane, each lane issuing all U of its
// loads of a batch (clamped to the plane) before it adds any of them, so that
// a wave keeps U KB in flight.
template <typename T, int U>
__global__ void __launch_bounds__(256)
k_pool_planes(const T* __restrict__ x, float* __restrict__ d, int64_t planes, int HW) {
  constexpr int EPV = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int nvec = HW / EPV;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t pl = wave; pl < planes; pl += nwaves) {
    const uint4* vb = reinterpret_cast<const uint4*>(x + pl * HW);
    float sum = 0.f;
    for (int v0 = 0; v0 < nvec; v0 += U * 64) {
      uint4 buf[U];
#pragma unroll
      for (int u = 0; u < U; ++u) buf[u] = vb[min(v0 + u * 64 + lane, nvec - 1)];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (v0 + u * 64 + lane < nvec) sum += sum16<T>(buf[u]);
    }
    sum = wave_sum<64>(sum);
    if (lane == 0) d[pl] = sum / (float)HW;
  }
}

// bf16 planes of a multiple of 4 positions: L lanes per plane (pool_rows.h)
template <int L>
__global__ void __launch_bounds__(256)
k_pool_nchw8(const uint16_t* __restrict__ x, float* __restrict__ d, int64_t planes, int HW) {
  const int64_t group = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / L;
  const int64_t ngroups = ((int64_t)gridDim.x * blockDim.x) / L;
  pool_planes8<L>(x, d, planes, HW, group, ngroups);
}

// grid B * nblk (nblk = ceil(vectors per row / 64)), block 256.  EPV channels per lane.
template <typename T, int EPV>
__global__ void __launch_bounds__(256)
k_pool_nhwc(const T* __restrict__ x, float* __restrict__ d, int C, int HW, int nblk) {
  __shared__ float part[4][64][EPV];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int64_t b = blockIdx.x / nblk;
  const int c0 = ((int)(blockIdx.x % nblk) * 64 + lane) * EPV;
  float acc[EPV];
#pragma unroll
  for (int j = 0; j < EPV; ++j) acc[j] = 0.f;
  if (c0 < C) {
    const T* img = x + (int64_t)b * HW * C + c0;
    for (int p = wv; p < HW; p += 4) {
      const T* row = img + (int64_t)p * C;
      if constexpr (EPV * sizeof(T) == 16) {
        const uint4 v = *reinterpret_cast<const uint4*>(row);
        if constexpr (sizeof(T) == 2) {
          acc[0] += bf16_lo(v.x); acc[1] += bf16_hi(v.x);
          acc[2] += bf16_lo(v.y); acc[3] += bf16_hi(v.y);
          acc[4] += bf16_lo(v.z); acc[5] += bf16_hi(v.z);
          acc[6] += bf16_lo(v.w); acc[7] += bf16_hi(v.w);
        } else {
          acc[0] += __uint_as_float(v.x); acc[1] += __uint_as_float(v.y);
          acc[2] += __uint_as_float(v.z); acc[3] += __uint_as_float(v.w);
        }
      } else {
#pragma unroll
        for (int j = 0; j < EPV; ++j) acc[j] += load_elem<T>(row + j);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < EPV; ++j) part[wv][lane][j] = acc[j];
  __syncthreads();
  if (wv == 0 && c0 < C) {
#pragma unroll
    for (int j = 0; j < EPV; ++j) {
      const float t = (part[0][lane][j] + part[1][lane][j]) + (part[2][lane][j] + part[3][lane][j]);
      if (c0 + j < C) d[(int64_t)b * C + c0 + j] = t / (float)HW;
    }
  }
}

template <typename T>
hipError_t pool_nchw(const Shape& sh, const T* x, float* d, hipStream_t st) {
  constexpr int EPV = 16 / sizeof(T);
  const int64_t planes = sh.B * sh.C;
  const int64_t nvec = sh.HW / EPV;
  if (sh.HW % EPV == 0 && nvec >= 256) {
    int64_t blocks = std::min<int64_t>((planes + 3) / 4, (int64_t)1 << 30);
    if (nvec <= 7 * 64) {
      // planes of at most 7 KB (the ResNet-50 stage-1 image: 6272 bytes): a
      // wave per plane, every vector loaded in one round of 7 per lane (0.4 us
      // faster at stage 1 than 8-load rounds over a capped grid)
      hipLaunchKernelGGL((k_pool_planes<T, 7>), dim3(blocks), dim3(256), 0, st, x, d, planes, (int)sh.HW);
      return hipGetLastError();
    }
    // longer planes: 8 loads per lane in flight, at most 8 workgroups per CU
    // and round
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL((k_pool_planes<T, 8>), dim3(blocks), dim3(256), 0, st, x, d, planes, (int)sh.HW);
    return hipGetLastError();
  }
  if constexpr (sizeof(T) == 2) {
    if (sh.HW % 4 == 0) {
      const int L8 = planes8_lanes(sh.HW);
      int64_t blocks8 = (planes + 256 / L8 - 1) / (256 / L8);
      if (blocks8 > 65536) blocks8 = 65536;
      const int HW = (int)sh.HW;
      switch (L8) {
        case 64: hipLaunchKernelGGL((k_pool_nchw8<64>), dim3(blocks8), dim3(256), 0, st, x, d, planes, HW); break;
        case 32: hipLaunchKernelGGL((k_pool_nchw8<32>), dim3(blocks8), dim3(256), 0, st, x, d, planes, HW); break;
        case 16: hipLaunchKernelGGL((k_pool_nchw8<16>), dim3(blocks8), dim3(256), 0, st, x, d, planes, HW); break;
        default: hipLaunchKernelGGL((k_pool_nchw8<8>), dim3(blocks8), dim3(256), 0, st, x, d, planes, HW); break;
      }
      return hipGetLastError();
    }
  }
  int L = nvec >= 128 ? 64 : nvec >= 48 ? 32 : nvec >= 16 ? 16 : 8;
  const int64_t groups_per_block = 256 / L;
  int64_t blocks = (planes + groups_per_block - 1) / groups_per_block;
  if (blocks > 65536) blocks = 65536;
  const int HW = (int)sh.HW;
  switch (L) {
    case 64: hipLaunchKernelGGL((k_pool_nchw<T, 64>), dim3(blocks), dim3(256), 0, st, x, d, planes, HW); break;
    case 32: hipLaunchKernelGGL((k_pool_nchw<T, 32>), dim3(blocks), dim3(256), 0, st, x, d, planes, HW); break;
    case 16: hipLaunchKernelGGL((k_pool_nchw<T, 16>), dim3(blocks), dim3(256), 0, st, x, d, planes, HW); break;
    default: hipLaunchKernelGGL((k_pool_nchw<T, 8>), dim3(blocks), dim3(256), 0, st, x, d, planes, HW); break;
  }
  return hipGetLastError();
}

// kPoolThreads threads per (image, block of 32 16-byte channel vectors)
template <typename T>
__global__ void __launch_bounds__(kPoolThreads)
k_pool_nhwc_rows(const T* __restrict__ x, float* __restrict__ d, int C, int HW, int nblk) {
  __shared__ float part[kPoolGroups * 32 * PoolVec<T>::EPV];
  pool_rows_block<T>(x, d, C, HW, blockIdx.x / nblk, blockIdx.x % nblk, part, C, 1);
}

template <typename T>
hipError_t pool_nhwc(const Shape& sh, const T* x, float* d, hipStream_t st) {
  constexpr int EPV16 = 16 / sizeof(T);
  const int C = (int)sh.C, HW = (int)sh.HW;
  if ((sh.C * sizeof(T)) % 16 == 0) {
    // every 16-byte vector of a row block read by its own lane, 32 row groups
    // with four loads in flight each
    const int nblk = (C / EPV16 + 31) / 32;
    hipLaunchKernelGGL((k_pool_nhwc_rows<T>), dim3((unsigned)(sh.B * nblk)), dim3(kPoolThreads), 0, st, x, d, C,
                       HW, nblk);
    return hipGetLastError();
  }
  const int nblk = (C + 63) / 64;
  hipLaunchKernelGGL((k_pool_nhwc<T, 1>), dim3((unsigned)(sh.B * nblk)), dim3(256), 0, st, x, d, C, HW, nblk);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pool(const Shape& sh, const void* x, float* d, hipStream_t st) {
  if (sh.layout == MOCE_NCHW) {
    return sh.elem == MOCE_F32 ? pool_nchw(sh, static_cast<const float*>(x), d, st)
                               : pool_nchw(sh, static_cast<const uint16_t*>(x), d, st);
  }
  return sh.elem == MOCE_F32 ? pool_nhwc(sh, static_cast<const float*>(x), d, st)
                             : pool_nhwc(sh, static_cast<const uint16_t*>(x), d, st);
}

}  // namespace moce

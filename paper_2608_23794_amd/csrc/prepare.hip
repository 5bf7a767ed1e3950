// Static support preparation (Sec. 3.2 Eq. 2 fixed at inference, Sec. 3.3
// gate input order, Sec. 3.4 uncovered set U).  Integer work; the result is
// unique, so every output is reproducible bit for bit.
#include <climits>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kPrepThreads = 256;

// Clears the coverage mask and seeds info = {0, INT_MAX}.
__global__ void k_prepare_clear(uint8_t* covered, int64_t C, int32_t* info) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i < C; i += (int64_t)gridDim.x * blockDim.x) covered[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    info[0] = 0;
    info[1] = INT_MAX;
  }
}

// One workgroup per routed expert row.  Each element's canonical position is
// its rank under "larger logit first, equal logits by lower channel"; one
// O(k^2) sweep also detects repeated channels.  Invalid rows report their
// index through an atomic minimum and write nothing.
// Idx: int32_t, or uint16_t for the 16-bit storage of deployed supports.
template <typename Idx>
__global__ void __launch_bounds__(kPrepThreads)
k_prepare_rows(const Idx* __restrict__ s, const float* __restrict__ w, int32_t* __restrict__ s_out,
               float* __restrict__ w_out, uint8_t* __restrict__ covered, int32_t* info, int C, int k) {
  extern __shared__ unsigned char smem[];
  int32_t* rs = reinterpret_cast<int32_t*>(smem);
  float* rw = reinterpret_cast<float*>(rs + k);
  __shared__ int bad;

  const int o = blockIdx.x;
  if (threadIdx.x == 0) bad = 0;
  for (int i = threadIdx.x; i < k; i += blockDim.x) {
    rs[i] = (int32_t)s[(int64_t)o * k + i];
    rw[i] = w[(int64_t)o * k + i];
  }
  __syncthreads();

  for (int i = threadIdx.x; i < k; i += blockDim.x) {
    const int32_t ci = rs[i];
    const float wi = rw[i];
    if (ci < 0 || ci >= C || !isfinite(wi)) bad = 1;
    for (int j = 0; j < k; ++j) {
      if (j != i && rs[j] == ci) bad = 1;
    }
  }
  __syncthreads();
  if (bad) {
    if (threadIdx.x == 0) atomicMin(&info[1], o);
    return;
  }

  for (int i = threadIdx.x; i < k; i += blockDim.x) {
    const int32_t ci = rs[i];
    const float wi = rw[i];
    int rank = 0;
    for (int j = 0; j < k; ++j) {
      const float wj = rw[j];
      rank += (wj > wi) || (wj == wi && rs[j] < ci);
    }
    s_out[(int64_t)o * k + rank] = ci;
    w_out[(int64_t)o * k + rank] = wi;
    covered[ci] = 1;
  }
}

// Single workgroup: ascending list of uncovered channels by a block-wide
// exclusive scan over chunks of the mask, then the final info values.
__global__ void __launch_bounds__(1024)
k_prepare_compact(const uint8_t* __restrict__ covered, int64_t C, int32_t* __restrict__ U, int32_t* info) {
  __shared__ int wave_tot[16];
  __shared__ int base;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  if (threadIdx.x == 0) base = 0;
  __syncthreads();
  for (int64_t c0 = 0; c0 < C; c0 += blockDim.x) {
    const int64_t c = c0 + threadIdx.x;
    const int flag = (c < C && !covered[c]) ? 1 : 0;
    const uint64_t ballot = __ballot(flag);
    const int before = __popcll(ballot & ((1ull << lane) - 1ull));
    if (lane == 0) wave_tot[wid] = __popcll(ballot);
    __syncthreads();
    int off = base;
    for (int q = 0; q < wid; ++q) off += wave_tot[q];
    if (flag) U[off + before] = (int32_t)c;
    __syncthreads();
    if (threadIdx.x == 0) {
      int tot = 0;
      for (int q = 0; q < nwaves; ++q) tot += wave_tot[q];
      base += tot;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    info[0] = base;
    if (info[1] == INT_MAX) info[1] = -1;
  }
}

}  // namespace

hipError_t launch_prepare(const Shape& sh, const void* s, bool s16, const float* w, int32_t* s_out,
                          float* w_out, uint8_t* covered, int32_t* U, int32_t* info,
                          hipStream_t st) {
  const int64_t C = sh.C;
  int clear_blocks = (int)((C + 255) / 256);
  if (clear_blocks > 4096) clear_blocks = 4096;
  if (clear_blocks < 1) clear_blocks = 1;
  hipLaunchKernelGGL(k_prepare_clear, dim3(clear_blocks), dim3(256), 0, st, covered, C, info);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (sh.R > 0) {
    const size_t lds = (size_t)sh.k * (sizeof(int32_t) + sizeof(float));
    if (s16)
      hipLaunchKernelGGL(k_prepare_rows<uint16_t>, dim3(sh.R), dim3(kPrepThreads), lds, st,
                         static_cast<const uint16_t*>(s), w, s_out, w_out, covered, info, (int)C, sh.k);
    else
      hipLaunchKernelGGL(k_prepare_rows<int32_t>, dim3(sh.R), dim3(kPrepThreads), lds, st,
                         static_cast<const int32_t*>(s), w, s_out, w_out, covered, info, (int)C, sh.k);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_prepare_compact, dim3(1), dim3(1024), 0, st, covered, C, U, info);
  return hipGetLastError();
}

}  // namespace moce

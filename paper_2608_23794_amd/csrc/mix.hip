// Routed experts (Sec. 3.3 Eq. 5) and the residual expert (Sec. 3.4 Eq. 6).
//
// NCHW: a block owns one tile of T = 64*PPL consecutive positions of one
// image and stages that tile of every input channel in LDS once
// ([C][T], input element type).  Each wave then takes whole output channels:
// lanes hold PPL consecutive positions, the support index and the coefficient
// are wave-uniform (scalar loads), and every LDS read is a contiguous,
// conflict-free row segment.  Each staged channel is reused by every expert
// whose support holds it.  The residual expert is one more output channel
// whose "support" is U with weights 1/|U|.
//
// NHWC: a block owns TP positions of one image, staged transposed into LDS as
// float32 [C][TP] so that one lane (one output channel) reads the TP values of
// a support channel as contiguous 16-byte loads.  Output rows y[b][p][:] are
// written with consecutive lanes on consecutive channels.
//
// Coefficients come from alpha[b][o][i] or are rebuilt from the logits and
// the softmax statistics of (b, o) with the gate kernel's operations.
#include "moce_internal.h"

namespace moce {
namespace {

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static float load(const float* p) { return *p; }
  __device__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<uint16_t> {
  __device__ static float load(const uint16_t* p) { return bf16_to_f32(*p); }
  __device__ static void store(uint16_t* p, float v) { *p = f32_to_bf16(v); }
};

// PPL consecutive elements of one LDS row, widened to float.
template <typename T, int PPL> struct Row;
template <> struct Row<uint16_t, 1> {
  __device__ static void get(const uint16_t* p, float* v) { v[0] = bf16_to_f32(*p); }
};
template <> struct Row<uint16_t, 2> {
  __device__ static void get(const uint16_t* p, float* v) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    v[0] = bf16_lo(u); v[1] = bf16_hi(u);
  }
};
template <> struct Row<uint16_t, 4> {
  __device__ static void get(const uint16_t* p, float* v) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    v[0] = bf16_lo(u.x); v[1] = bf16_hi(u.x); v[2] = bf16_lo(u.y); v[3] = bf16_hi(u.y);
  }
};
template <> struct Row<float, 1> {
  __device__ static void get(const float* p, float* v) { v[0] = *p; }
};
template <> struct Row<float, 2> {
  __device__ static void get(const float* p, float* v) {
    const float2 u = *reinterpret_cast<const float2*>(p); v[0] = u.x; v[1] = u.y;
  }
};
template <> struct Row<float, 4> {
  __device__ static void get(const float* p, float* v) {
    const float4 u = *reinterpret_cast<const float4*>(p); v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
};

// PPL consecutive outputs of one lane; the address is PPL-element aligned.
template <typename T, int PPL> struct RowStore {
  __device__ static void put(T* p, const float* v) {
#pragma unroll
    for (int j = 0; j < PPL; ++j) Elem<T>::store(p + j, v[j]);
  }
};
template <> struct RowStore<uint16_t, 2> {
  __device__ static void put(uint16_t* p, const float* v) {
    *reinterpret_cast<uint32_t*>(p) = pack_bf16x2(v[0], v[1]);
  }
};
template <> struct RowStore<uint16_t, 4> {
  __device__ static void put(uint16_t* p, const float* v) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
};
template <> struct RowStore<float, 2> {
  __device__ static void put(float* p, const float* v) { *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]); }
};
template <> struct RowStore<float, 4> {
  __device__ static void put(float* p, const float* v) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

template <int VB> struct VecOf;
template <> struct VecOf<16> { using type = uint4; };
template <> struct VecOf<8> { using type = uint2; };
template <> struct VecOf<4> { using type = uint32_t; };
template <> struct VecOf<2> { using type = uint16_t; };

// Coefficient source for expert o of image b: alpha as given, or rebuilt
// from the logits and the softmax statistics with the gate's operations
// (bit-identical to the coefficients the gate kernel writes).
template <bool ALPHA> struct Coef;
template <> struct Coef<true> {
  const float* row;
  __device__ Coef(const float* alpha, const float*, const float*, int64_t, int64_t bo, int o, int k)
      : row(alpha + bo * k) {}
  __device__ float operator()(int i) const { return row[i]; }
};
template <> struct Coef<false> {
  const float* wo;
  float rt, m, rzs;
  __device__ Coef(const float*, const float* w, const float* st, int64_t n, int64_t bo, int o, int k)
      : wo(w + (int64_t)o * k), rt(st[bo]), m(st[n + bo]), rzs(st[2 * n + bo]) {}
  __device__ float operator()(int i) const { return coef_alpha(coef_e(coef_z(wo[i], rt), m), rzs); }
};

// ------------------------------------------------------------------ NCHW
template <typename T, int PPL, int NW, int VB, bool ALPHA>
__global__ void __launch_bounds__(NW * 64)
k_mix_nchw(const T* __restrict__ x, const int32_t* __restrict__ s, const float* __restrict__ alpha,
           const float* __restrict__ w, const float* __restrict__ st, int64_t nst,
           const int32_t* __restrict__ U, int nU, T* __restrict__ y, int C, int HW, int E, int R, int k,
           int tiles) {
  constexpr int TT = 64 * PPL;
  constexpr int EV = VB / (int)sizeof(T);
  constexpr int VPR = TT / EV;
  using V = typename VecOf<VB>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  T* tile = reinterpret_cast<T*>(smem);

  const int64_t b = blockIdx.x / tiles;
  const int p0 = (int)(blockIdx.x % tiles) * TT;
  const int valid = min(TT, HW - p0);
  const int vvalid = valid / EV;  // H*W*sizeof(T) is a multiple of VB, so valid is a multiple of EV

  const T* xb = x + b * C * HW + p0;
  for (int idx = threadIdx.x; idx < C * VPR; idx += NW * 64) {
    const int c = idx / VPR;
    const int v = idx - c * VPR;
    V val{};
    if (v < vvalid) val = *reinterpret_cast<const V*>(xb + (int64_t)c * HW + v * EV);
    *reinterpret_cast<V*>(tile + c * TT + v * EV) = val;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const T* trow = tile + lane * PPL;
  T* yb = y + b * (int64_t)E * HW + p0 + lane * PPL;
  const bool full = (lane + 1) * PPL <= valid;
  for (int o = wv; o < E; o += NW) {
    float acc[PPL];
#pragma unroll
    for (int j = 0; j < PPL; ++j) acc[j] = 0.f;
    if (o < R) {
      const int32_t* so = s + (int64_t)o * k;
      const Coef<ALPHA> coef(alpha, w, st, nst, b * R + o, o, k);
#pragma unroll 4
      for (int i = 0; i < k; ++i) {
        float v[PPL];
        Row<T, PPL>::get(trow + so[i] * TT, v);
        const float a = coef(i);
#pragma unroll
        for (int j = 0; j < PPL; ++j) acc[j] = fmaf(a, v[j], acc[j]);
      }
    } else if (nU > 0) {
#pragma unroll 4
      for (int u = 0; u < nU; ++u) {
        float v[PPL];
        Row<T, PPL>::get(trow + U[u] * TT, v);
#pragma unroll
        for (int j = 0; j < PPL; ++j) acc[j] += v[j];
      }
#pragma unroll
      for (int j = 0; j < PPL; ++j) acc[j] = acc[j] / (float)nU;
    }
    T* yo = yb + (int64_t)o * HW;
    if (full) {
      RowStore<T, PPL>::put(yo, acc);
    } else {
#pragma unroll
      for (int j = 0; j < PPL; ++j)
        if (lane * PPL + j < valid) Elem<T>::store(yo + j, acc[j]);
    }
  }
}

// Any shape: every read goes to global memory (lanes on consecutive positions).
template <typename T, bool ALPHA>
__global__ void __launch_bounds__(256)
k_mix_nchw_global(const T* __restrict__ x, const int32_t* __restrict__ s, const float* __restrict__ alpha,
                  const float* __restrict__ w, const float* __restrict__ st, int64_t nst,
                  const int32_t* __restrict__ U, int nU, T* __restrict__ y, int C, int HW, int E, int R, int k,
                  int tiles) {
  const int64_t b = blockIdx.x / tiles;
  const int p = (int)(blockIdx.x % tiles) * 64 + (threadIdx.x & 63);
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const T* xb = x + b * C * HW + p;
  for (int o = wv; o < E; o += 4) {
    float acc = 0.f;
    if (o < R) {
      const int32_t* so = s + (int64_t)o * k;
      const Coef<ALPHA> coef(alpha, w, st, nst, b * R + o, o, k);
      if (p < HW)
        for (int i = 0; i < k; ++i) acc = fmaf(coef(i), Elem<T>::load(xb + (int64_t)so[i] * HW), acc);
    } else if (nU > 0) {
      if (p < HW)
        for (int u = 0; u < nU; ++u) acc += Elem<T>::load(xb + (int64_t)U[u] * HW);
      acc = acc / (float)nU;
    }
    if (p < HW) Elem<T>::store(y + (b * E + o) * (int64_t)HW + p, acc);
  }
}

// ------------------------------------------------------------------ NHWC
// 64 NS threads; work item (expert o, part h < NS) computes o at positions
// h TP/NS .. h TP/NS + TP/NS - 1 of the tile, so each item's chain of index,
// LDS and FMA steps covers fewer products and NS times as many chains run.
template <typename T, int TP, int NS, bool ALPHA>
__global__ void __launch_bounds__(64 * NS * 4)
k_mix_nhwc(const T* __restrict__ x, const int32_t* __restrict__ s, const float* __restrict__ alpha,
           const float* __restrict__ w, const float* __restrict__ st, int64_t nst,
           const int32_t* __restrict__ U, int nU, T* __restrict__ y, int C, int HW, int E, int R, int k,
           int tiles) {
  static_assert(TP % (4 * NS) == 0, "a work item's positions are read as float4");
  extern __shared__ __align__(16) unsigned char smem[];
  float* tile = reinterpret_cast<float*>(smem);  // [C][TP]

  const int64_t b = blockIdx.x / tiles;
  const int p0 = (int)(blockIdx.x % tiles) * TP;
  const int valid = min(TP, HW - p0);
  const T* src = x + (b * HW + p0) * (int64_t)C;
  for (int idx = threadIdx.x; idx < TP * C; idx += blockDim.x) {
    const int p = idx / C;
    const int c = idx - p * C;
    tile[c * TP + p] = p < valid ? Elem<T>::load(src + idx) : 0.f;
  }
  __syncthreads();

  constexpr int TH = TP / NS;  // positions per work item
  T* yb = y + (b * HW + p0) * (int64_t)E;
  for (int it = threadIdx.x; it < NS * E; it += blockDim.x) {
    const int o = it / NS, h = it % NS;
    float acc[TH];
#pragma unroll
    for (int j = 0; j < TH; ++j) acc[j] = 0.f;
    if (o < R) {
      const int32_t* so = s + (int64_t)o * k;
      const Coef<ALPHA> coef(alpha, w, st, nst, b * R + o, o, k);
#pragma unroll 2
      for (int i = 0; i < k; ++i) {
        const float a = coef(i);
        const float4* r = reinterpret_cast<const float4*>(tile + so[i] * TP + h * TH);
#pragma unroll
        for (int q = 0; q < TH / 4; ++q) {
          const float4 v = r[q];
          acc[4 * q + 0] = fmaf(a, v.x, acc[4 * q + 0]);
          acc[4 * q + 1] = fmaf(a, v.y, acc[4 * q + 1]);
          acc[4 * q + 2] = fmaf(a, v.z, acc[4 * q + 2]);
          acc[4 * q + 3] = fmaf(a, v.w, acc[4 * q + 3]);
        }
      }
    } else if (nU > 0) {
      for (int u = 0; u < nU; ++u) {
        const float4* r = reinterpret_cast<const float4*>(tile + U[u] * TP + h * TH);
#pragma unroll
        for (int q = 0; q < TH / 4; ++q) {
          const float4 v = r[q];
          acc[4 * q + 0] += v.x; acc[4 * q + 1] += v.y; acc[4 * q + 2] += v.z; acc[4 * q + 3] += v.w;
        }
      }
#pragma unroll
      for (int j = 0; j < TH; ++j) acc[j] = acc[j] / (float)nU;
    }
#pragma unroll
    for (int j = 0; j < TH; ++j)
      if (h * TH + j < valid) Elem<T>::store(yb + (int64_t)(h * TH + j) * E + o, acc[j]);
  }
}

template <typename T, bool ALPHA>
__global__ void __launch_bounds__(256)
k_mix_nhwc_global(const T* __restrict__ x, const int32_t* __restrict__ s, const float* __restrict__ alpha,
                  const float* __restrict__ w, const float* __restrict__ st, int64_t nst,
                  const int32_t* __restrict__ U, int nU, T* __restrict__ y, int C, int HW, int E, int R, int k) {
  const int64_t b = blockIdx.x / HW;
  const int p = (int)(blockIdx.x % HW);
  const T* row = x + (b * HW + p) * (int64_t)C;
  for (int o = threadIdx.x; o < E; o += blockDim.x) {
    float acc = 0.f;
    if (o < R) {
      const int32_t* so = s + (int64_t)o * k;
      const Coef<ALPHA> coef(alpha, w, st, nst, b * R + o, o, k);
      for (int i = 0; i < k; ++i) acc = fmaf(coef(i), Elem<T>::load(row + so[i]), acc);
    } else if (nU > 0) {
      for (int u = 0; u < nU; ++u) acc += Elem<T>::load(row + U[u]);
      acc = acc / (float)nU;
    }
    Elem<T>::store(y + (b * HW + p) * (int64_t)E + o, acc);
  }
}

// ------------------------------------------------------------------ dispatch
constexpr size_t kLdsMax = 160 * 1024;

template <typename K>
void allow_lds(K kernel, size_t bytes) {
  if (bytes > 64 * 1024)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

struct MixArgs {
  const int32_t* s; const float* alpha; const float* w; const float* st;
  const int32_t* U; int nU;
};

template <typename T, int PPL, int VB, bool ALPHA>
hipError_t nchw_launch(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  // 16 waves, each through a chain of dependent index, LDS and FMA steps for
  // its experts: twice the chains in flight of 8 waves (ResNet-50 stage-3
  // NCHW mix 102 -> 61 us)
  constexpr int NW = 16;
  const int TT = 64 * PPL;
  const int tiles = (int)((sh.HW + TT - 1) / TT);
  const size_t lds = (size_t)sh.C * TT * sizeof(T);
  auto kern = k_mix_nchw<T, PPL, NW, VB, ALPHA>;
  allow_lds(kern, lds);
  hipLaunchKernelGGL(kern, dim3((unsigned)(sh.B * tiles)), dim3(NW * 64), lds, st, x, a.s, a.alpha, a.w,
                     a.st, sh.B * sh.R, a.U, a.nU, y, (int)sh.C, (int)sh.HW, sh.E, sh.R, sh.k, tiles);
  return hipGetLastError();
}

template <typename T, int PPL, bool ALPHA>
hipError_t nchw_pick_vec(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  const int64_t row_bytes = sh.HW * (int64_t)sizeof(T);
  if (row_bytes % 16 == 0) return nchw_launch<T, PPL, 16, ALPHA>(sh, x, y, a, st);
  if (row_bytes % 8 == 0) return nchw_launch<T, PPL, 8, ALPHA>(sh, x, y, a, st);
  if (row_bytes % 4 == 0) return nchw_launch<T, PPL, 4, ALPHA>(sh, x, y, a, st);
  if constexpr (sizeof(T) == 2) return nchw_launch<T, PPL, 2, ALPHA>(sh, x, y, a, st);
  return hipErrorInvalidValue;
}

template <typename T, bool ALPHA>
hipError_t mix_nchw(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  const size_t row1 = (size_t)sh.C * 64 * sizeof(T);
  const int64_t hw64 = (sh.HW + 63) / 64 * 64;
  if (row1 * 2 <= 64 * 1024 && hw64 >= 128 && sh.HW % 2 == 0) {
    if (row1 * 4 <= 64 * 1024 && hw64 >= 256 && sh.HW % 4 == 0)
      return nchw_pick_vec<T, 4, ALPHA>(sh, x, y, a, st);
    return nchw_pick_vec<T, 2, ALPHA>(sh, x, y, a, st);
  }
  if (row1 <= kLdsMax) return nchw_pick_vec<T, 1, ALPHA>(sh, x, y, a, st);
  const int tiles = (int)((sh.HW + 63) / 64);
  hipLaunchKernelGGL((k_mix_nchw_global<T, ALPHA>), dim3((unsigned)(sh.B * tiles)), dim3(256), 0, st, x, a.s,
                     a.alpha, a.w, a.st, sh.B * sh.R, a.U, a.nU, y, (int)sh.C, (int)sh.HW, sh.E, sh.R, sh.k, tiles);
  return hipGetLastError();
}

template <typename T, int TP, bool ALPHA>
hipError_t nhwc_launch(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  constexpr int NS = TP / 4;  // work items of 4 positions
  const size_t lds = (size_t)sh.C * TP * sizeof(float);
  const int tiles = (int)((sh.HW + TP - 1) / TP);
  auto kern = k_mix_nhwc<T, TP, NS, ALPHA>;
  allow_lds(kern, lds);
  hipLaunchKernelGGL(kern, dim3((unsigned)(sh.B * tiles)), dim3(256 * NS), lds, st, x, a.s, a.alpha, a.w, a.st,
                     sh.B * sh.R, a.U, a.nU, y, (int)sh.C, (int)sh.HW, sh.E, sh.R, sh.k, tiles);
  return hipGetLastError();
}

// 16 positions per workgroup where their float32 tile fits in LDS (10-14%
// faster than 8 at ResNet-50 stages 3 and 4 and the ViT token layer, whose
// inner loops are latency chains: each index and coefficient read then serves
// twice the products; 32 is slower), else 8, else the global-memory kernel.
template <typename T, bool ALPHA>
hipError_t mix_nhwc(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  if ((size_t)sh.C * 16 * sizeof(float) <= kLdsMax) return nhwc_launch<T, 16, ALPHA>(sh, x, y, a, st);
  if ((size_t)sh.C * 8 * sizeof(float) <= kLdsMax) return nhwc_launch<T, 8, ALPHA>(sh, x, y, a, st);
  hipLaunchKernelGGL((k_mix_nhwc_global<T, ALPHA>), dim3((unsigned)(sh.B * sh.HW)), dim3(256), 0, st, x, a.s,
                     a.alpha, a.w, a.st, sh.B * sh.R, a.U, a.nU, y, (int)sh.C, (int)sh.HW, sh.E, sh.R, sh.k);
  return hipGetLastError();
}

template <typename T>
hipError_t mix_typed(const Shape& sh, const T* x, T* y, const MixArgs& a, hipStream_t st) {
  if (sh.layout == MOCE_NCHW)
    return a.alpha ? mix_nchw<T, true>(sh, x, y, a, st) : mix_nchw<T, false>(sh, x, y, a, st);
  return a.alpha ? mix_nhwc<T, true>(sh, x, y, a, st) : mix_nhwc<T, false>(sh, x, y, a, st);
}

}  // namespace

hipError_t launch_mix(const Shape& sh, const void* x, const int32_t* s, const float* alpha,
                      const float* w, const float* stats, const int32_t* U, int nU,
                      void* y, hipStream_t st) {
  const MixArgs a{s, alpha, w, stats, U, nU};
  if (sh.elem == MOCE_F32)
    return mix_typed(sh, static_cast<const float*>(x), static_cast<float*>(y), a, st);
  return mix_typed(sh, static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y), a, st);
}

namespace {

// In place: y = act(scale[o] y + shift[o]) with o the output channel of each
// element, a thread per element.
template <typename T, bool NHWC>
__global__ void k_epilogue(T* __restrict__ y, int64_t n, int E, int64_t HW, Epi ep) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int o = NHWC ? (int)(i % E) : (int)((i / HW) % E);
    Elem<T>::store(y + i, epi_apply(ep, Elem<T>::load(y + i), o));
  }
}

}  // namespace

hipError_t launch_epilogue(const Shape& sh, void* y, const Epi& ep, hipStream_t st) {
  if (!epi_active(ep)) return hipSuccess;
  const int64_t n = sh.B * sh.E * sh.HW;
  const unsigned grid = (unsigned)std::min<int64_t>((n + 255) / 256, 65536);
  const bool nhwc = sh.layout == MOCE_NHWC;
  if (sh.elem == MOCE_BF16) {
    auto p = static_cast<uint16_t*>(y);
    if (nhwc)
      k_epilogue<uint16_t, true><<<grid, 256, 0, st>>>(p, n, sh.E, sh.HW, ep);
    else
      k_epilogue<uint16_t, false><<<grid, 256, 0, st>>>(p, n, sh.E, sh.HW, ep);
  } else {
    auto p = static_cast<float*>(y);
    if (nhwc)
      k_epilogue<float, true><<<grid, 256, 0, st>>>(p, n, sh.E, sh.HW, ep);
    else
      k_epilogue<float, false><<<grid, 256, 0, st>>>(p, n, sh.E, sh.HW, ep);
  }
  return hipGetLastError();
}

}  // namespace moce

// Temperatures (Sec. 3.3) and mixing coefficients (Sec. 3.3 Eq. 4).
//
// One wavefront, or a 32- or 16-lane segment, per (image, routed expert).
// Lanes span the k support positions: each gathers the descriptor of its
// channel, the segment reduces the gate's pre-activation, and the same lanes
// then form the softmax of the selected logits over the temperature with the
// library's coefficient operations (coef_z, coef_e, coef_alpha).  Optionally
// writes the coefficients alpha[b][o][i] and/or the softmax statistics
// (rt = 1/tau, the largest scaled logit m, rzs = 1 / partition sum), from
// which a mix kernel rebuilds exactly the same coefficients.
#include <type_traits>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kGateWaves = 4;

__device__ __forceinline__ void put_stats(const Stats& st, int64_t item, float rt, float m, float rzs) {
  st.rt[item] = rt;
  st.m[item] = m;
  st.rzs[item] = rzs;
}

__device__ __forceinline__ void softmax_epilogue(const float* __restrict__ wo, int k, float t, int lane,
                                                 float* __restrict__ alpha_row, const Stats* st, int64_t item) {
  const float rt = 1.f / t;
  float m = -INFINITY;
  for (int i = lane; i < k; i += kWave) m = fmaxf(m, coef_z(wo[i], rt));
  m = wave_max(m);
  float z = 0.f;
  for (int i = lane; i < k; i += kWave) z += coef_e(coef_z(wo[i], rt), m);
  z = wave_sum(z);
  const float rzs = 1.f / z;
  if (alpha_row) {
    for (int i = lane; i < k; i += kWave) alpha_row[i] = coef_alpha(coef_e(coef_z(wo[i], rt), m), rzs);
  }
  if (st && lane == 0) put_stats(*st, item, rt, m, rzs);
}

__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_softplus(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                float* __restrict__ alpha, Stats st, int64_t B, int64_t C, int R, int k) {
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * kGateWaves + (threadIdx.x >> 6);
  if (item >= B * R) return;
  const int64_t b = item / R;
  const int o = (int)(item % R);
  const int32_t* so = s + (int64_t)o * k;
  const float* ao = a + (int64_t)o * k;
  const float* db = d + b * C;
  float g = 0.f;
  for (int i = lane; i < k; i += kWave) g += ao[i] * db[so[i]];
  g = wave_sum(g) + c[o];
  const float t = softplusf(g) + 1e-3f;
  if (lane == 0) tau[item] = t;
  softmax_epilogue(w + (int64_t)o * k, k, t, lane, alpha ? alpha + item * k : nullptr, st.rt ? &st : nullptr,
                   item);
}

// The same for k <= W (W = 32): segments of W lanes, one per (image,
// expert), 64 / W per wave, lane i of a segment holding support position i.
// Every input of a position is read up front (the selected logit too), so the
// only dependent reads are the descriptor gathers; the exponentials are
// formed once and reused for the coefficients.
template <int W>
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_softplus_seg(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                    const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                    float* __restrict__ alpha, Stats st, int64_t B, int64_t C, int R, int k) {
  constexpr int kSeg = kWave / W;
  const int lane = threadIdx.x & 63;
  const int i = lane & (W - 1);
  const int64_t item = ((int64_t)blockIdx.x * kGateWaves + (threadIdx.x >> 6)) * kSeg + lane / W;
  const bool live = item < B * R;
  const int64_t it = live ? item : B * R - 1;
  const int64_t b = it / R;
  const int o = (int)(it % R);
  const bool in = i < k;
  const int64_t e = (int64_t)o * k + (in ? i : 0);
  const int ch = s[e];
  const float av = a[e];
  const float wv = w[e];
  const float co = c[o];
  float g = in ? av * d[b * C + ch] : 0.f;
  g = wave_sum<W>(g) + co;
  const float t = softplusf(g) + 1e-3f;
  const float rt = 1.f / t;
  const float z = coef_z(wv, rt);
  const float m = wave_max<W>(in ? z : -INFINITY);
  const float ex = in ? coef_e(z, m) : 0.f;
  const float zs = wave_sum<W>(ex);
  const float rzs = 1.f / zs;
  if (!live) return;
  if (i == 0) tau[item] = t;
  if (alpha && in) alpha[item * k + i] = coef_alpha(ex, rzs);
  if (st.rt && i == 0) put_stats(st, item, rt, m, rzs);
}

// The value of lane l ^ OFF within rows of 16 lanes, by DPP moves (quad
// permutations, row shifts, a half-row rotation).
template <int OFF>
__device__ __forceinline__ float row16_xor(float v, int lane) {
  auto mov = [](float u, auto ctrl) __attribute__((always_inline)) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(u), decltype(ctrl)::value, 0xf, 0xf, true));
  };
  if constexpr (OFF == 1) {
    return mov(v, std::integral_constant<int, 0xb1>{});  // quad_perm [1, 0, 3, 2]
  } else if constexpr (OFF == 2) {
    return mov(v, std::integral_constant<int, 0x4e>{});  // quad_perm [2, 3, 0, 1]
  } else if constexpr (OFF == 4) {
    const float up = mov(v, std::integral_constant<int, 0x104>{});  // row_shl 4: lane l + 4
    const float dn = mov(v, std::integral_constant<int, 0x114>{});  // row_shr 4: lane l - 4
    return (lane & 4) ? dn : up;
  } else {
    return mov(v, std::integral_constant<int, 0x128>{});  // row_ror 8: lane l ^ 8 within the row
  }
}
__device__ __forceinline__ float row16_sum(float v, int lane) {
  v += row16_xor<8>(v, lane);
  v += row16_xor<4>(v, lane);
  v += row16_xor<2>(v, lane);
  v += row16_xor<1>(v, lane);
  return v;
}
__device__ __forceinline__ float row16_max(float v, int lane) {
  v = fmaxf(v, row16_xor<8>(v, lane));
  v = fmaxf(v, row16_xor<4>(v, lane));
  v = fmaxf(v, row16_xor<2>(v, lane));
  v = fmaxf(v, row16_xor<1>(v, lane));
  return v;
}

// The softplus-linear gate for 32 < k <= 16 PER: a row of 16 lanes per
// (image, expert), four per wave, lane h holding support positions
// h, h + 16, ..., so that each read instruction covers 16 consecutive entries
// of every pair.  Every input of a lane is read up front; the three
// reductions are DPP moves within the row.
template <int PER>
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_softplus_x16(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                    const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                    float* __restrict__ alpha, Stats st, int64_t B, int64_t C, int R, int k) {
  const int lane = threadIdx.x & 63;
  const int h = lane & 15;
  const int64_t item = ((int64_t)blockIdx.x * kGateWaves + (threadIdx.x >> 6)) * 4 + (lane >> 4);
  const bool live = item < B * R;
  const int64_t it = live ? item : B * R - 1;
  const int64_t b = it / R;
  const int o = (int)(it % R);
  const int64_t e0 = (int64_t)o * k;
  int ch[PER];
  float av[PER], wv[PER], dv[PER];
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    const int i = min(h + 16 * t, k - 1);
    ch[t] = s[e0 + i];
    av[t] = a[e0 + i];
    wv[t] = w[e0 + i];
  }
  const float co = c[o];
  const float* db = d + b * C;
#pragma unroll
  for (int t = 0; t < PER; ++t) dv[t] = db[ch[t]];
  float g = 0.f;
#pragma unroll
  for (int t = 0; t < PER; ++t)
    if (h + 16 * t < k) g += av[t] * dv[t];
  g = row16_sum(g, lane) + co;
  const float tv = softplusf(g) + 1e-3f;
  const float rt = 1.f / tv;
  float z[PER];
  float m = -INFINITY;
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    z[t] = coef_z(wv[t], rt);
    if (h + 16 * t < k) m = fmaxf(m, z[t]);
  }
  m = row16_max(m, lane);
  float zs = 0.f;
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    z[t] = coef_e(z[t], m);
    if (h + 16 * t < k) zs += z[t];
  }
  zs = row16_sum(zs, lane);
  const float rzs = 1.f / zs;
  if (!live) return;
  if (h == 0) tau[item] = tv;
  if (alpha) {
#pragma unroll
    for (int t = 0; t < PER; ++t)
      if (h + 16 * t < k) alpha[item * k + h + 16 * t] = coef_alpha(z[t], rzs);
  }
  if (st.rt && h == 0) put_stats(st, item, rt, m, rzs);
}

// The paper's shared gate: h = ReLU(W1 z + b1), g = w2 . h + b2,
// tau = tau_min + (tau_max - tau_min) sigmoid(g).  k <= 256 (4 hidden units
// per lane at most).
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_mlp(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
           const float* __restrict__ W1, const float* __restrict__ b1, const float* __restrict__ w2,
           float b2, float tau_min, float tau_max, float* __restrict__ tau, float* __restrict__ alpha,
           Stats st, int64_t B, int64_t C, int R, int k) {
  __shared__ float zs[kGateWaves][256];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int64_t item = (int64_t)blockIdx.x * kGateWaves + wv;
  const bool active = item < B * R;  // every wave reaches the barrier below
  const int64_t b = active ? item / R : 0;
  const int o = active ? (int)(item % R) : 0;
  const int32_t* so = s + (int64_t)o * k;
  for (int i = lane; i < k; i += kWave) zs[wv][i] = d[b * C + so[i]];
  __syncthreads();
  if (!active) return;
  float g = 0.f;
  for (int j = lane; j < k; j += kWave) {
    const float* row = W1 + (int64_t)j * k;
    float h = b1[j];
    for (int i = 0; i < k; ++i) h += row[i] * zs[wv][i];
    g += w2[j] * fmaxf(h, 0.f);
  }
  g = wave_sum(g) + b2;
  const float t = tau_min + (tau_max - tau_min) / (1.f + expf(-g));
  if (lane == 0) tau[item] = t;
  softmax_epilogue(w + (int64_t)o * k, k, t, lane, alpha ? alpha + item * k : nullptr, st.rt ? &st : nullptr,
                   item);
}

}  // namespace

hipError_t launch_gate(const Shape& sh, const float* d, const int32_t* s, const float* w,
                       const moce_gate_params& g, float* tau, float* alpha, float* stats, hipStream_t st) {
  if (sh.R == 0) return hipSuccess;
  const int64_t items = sh.B * sh.R;
  const Stats sp = stats ? stats_planes(stats, items) : Stats{nullptr, nullptr, nullptr};
  const unsigned blocks = (unsigned)((items + kGateWaves - 1) / kGateWaves);
  if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 32) {
    const unsigned b32 = (unsigned)((items + 2 * kGateWaves - 1) / (2 * kGateWaves));
    hipLaunchKernelGGL(k_gate_softplus_seg<32>, dim3(b32), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 256) {
    // rows of 16 lanes, four (image, expert) pairs per wave
    const unsigned b16 = (unsigned)((items + 4 * kGateWaves - 1) / (4 * kGateWaves));
    const int per = (sh.k + 15) / 16;
    auto kern = per <= 4 ? k_gate_softplus_x16<4> : per <= 8 ? k_gate_softplus_x16<8> : k_gate_softplus_x16<16>;
    hipLaunchKernelGGL(kern, dim3(b16), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c, tau, alpha, sp, sh.B,
                       sh.C, sh.R, sh.k);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR) {
    hipLaunchKernelGGL(k_gate_softplus, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  } else {
    hipLaunchKernelGGL(k_gate_mlp, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.W1, g.b1, g.w2,
                       g.b2, g.tau_min, g.tau_max, tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  }
  return hipGetLastError();
}

}  // namespace moce

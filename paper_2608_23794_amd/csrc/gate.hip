// Temperatures (Sec. 3.3) and mixing coefficients (Sec. 3.3 Eq. 4).
//
// One wavefront (or a 32- or 64-lane segment) per (image, routed expert).
// Lanes span the k support positions: each gathers the descriptor of its
// channel, the segment reduces the gate's pre-activation, and the same lanes
// then form the softmax of the selected logits over the temperature with the
// library's coefficient operations (coef_z, coef_e, coef_alpha).  Optionally
// writes the coefficients alpha[b][o][i] and/or the softmax statistics
// (rt = 1/tau, the largest scaled logit m, rzs = 1 / partition sum), from
// which a mix kernel rebuilds exactly the same coefficients.
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

// The same for 64 < k <= 64 PER: every input of a lane's PER positions is
// read up front (indices, slopes and logits, then the descriptor gathers),
// so the wave makes two dependent round trips instead of one per pass, and
// the quotients are kept for the three reductions.  The operations and their
// order per lane are those of k_gate_softplus.
template <int PER>
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_softplus_wide(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                     const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                     float* __restrict__ alpha, Stats st, int64_t B, int64_t C, int R, int k) {
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * kGateWaves + (threadIdx.x >> 6);
  if (item >= B * R) return;
  const int64_t b = item / R;
  const int o = (int)(item % R);
  const int32_t* so = s + (int64_t)o * k;
  const float* ao = a + (int64_t)o * k;
  const float* wo = w + (int64_t)o * k;
  const float* db = d + b * C;
  int ch[PER];
  float av[PER], wv[PER], dv[PER];
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int i = min(lane + kWave * r, k - 1);
    ch[r] = so[i];
    av[r] = ao[i];
    wv[r] = wo[i];
  }
#pragma unroll
  for (int r = 0; r < PER; ++r) dv[r] = db[ch[r]];
  float g = 0.f;
#pragma unroll
  for (int r = 0; r < PER; ++r)
    if (lane + kWave * r < k) g += av[r] * dv[r];
  g = wave_sum(g) + c[o];
  const float t = softplusf(g) + 1e-3f;
  if (lane == 0) tau[item] = t;
  const float rt = 1.f / t;
  float z[PER];
  float m = -INFINITY;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    z[r] = coef_z(wv[r], rt);
    if (lane + kWave * r < k) m = fmaxf(m, z[r]);
  }
  m = wave_max(m);
  float zs = 0.f;
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    z[r] = coef_e(z[r], m);
    if (lane + kWave * r < k) zs += z[r];
  }
  zs = wave_sum(zs);
  const float rzs = 1.f / zs;
  if (alpha) {
#pragma unroll
    for (int r = 0; r < PER; ++r)
      if (lane + kWave * r < k) alpha[item * k + lane + kWave * r] = coef_alpha(z[r], rzs);
  }
  if (st.rt && lane == 0) put_stats(st, item, rt, m, rzs);
}

// The same for k <= W (W = 32 or 64): segments of W lanes, one per (image,
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
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 64) {
    hipLaunchKernelGGL(k_gate_softplus_seg<64>, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 128) {
    hipLaunchKernelGGL(k_gate_softplus_wide<2>, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 256) {
    hipLaunchKernelGGL(k_gate_softplus_wide<4>, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
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

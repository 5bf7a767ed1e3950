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
#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kGateWaves = 4;
constexpr int64_t kGateTargetWaves = 4096;  // waves of the image-walking gate (16 per CU)
constexpr int64_t kLdsGateTargetBlocks = 512;  // workgroups of the LDS gate (two per CU)
constexpr int64_t kLdsGateMaxImages = 32;     // images per workgroup at most

__device__ __forceinline__ void put_stats(const Stats& st, int64_t b, int o, float rt, float m, float rzs) {
  const int64_t i = b * st.sb + o * st.so;
  st.rt[i] = rt;
  st.m[i] = m;
  st.rzs[i] = rzs;
}

__device__ __forceinline__ void softmax_epilogue(const float* __restrict__ wo, int k, float t, int lane,
                                                 float* __restrict__ alpha_row, const Stats* st, int64_t b, int o) {
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
  if (st && lane == 0) put_stats(*st, b, o, rt, m, rzs);
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
  softmax_epilogue(w + (int64_t)o * k, k, t, lane, alpha ? alpha + item * k : nullptr, st.rt ? &st : nullptr, b,
                   o);
}

// The same for k <= W (W = 8, 16 or 32): segments of W lanes, one per (image,
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
  if (st.rt && i == 0) put_stats(st, b, o, rt, m, rzs);
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
// routed expert, four experts per wave, lane h holding support positions
// h, h + 16, ..., so that each read instruction covers 16 consecutive entries
// of every expert.  A wave keeps its experts' supports, gate weights and
// logits in registers and walks `nbi` consecutive images, reading the next
// image's descriptor gathers while it forms the current one's softmax; the
// three reductions are DPP moves within the row.  Waves of one workgroup
// share their images, so an image's descriptor is fetched once per CU.
template <int PER>
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_softplus_x16(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                    const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                    float* __restrict__ alpha, Stats st, int64_t B, int64_t C, int R, int k, int nrow, int nbi) {
  const int lane = threadIdx.x & 63;
  const int h = lane & 15;
  const int64_t wave = (int64_t)blockIdx.x * kGateWaves + (threadIdx.x >> 6);
  const int64_t b0 = (wave / nrow) * nbi;
  const int orow = (int)(wave % nrow);
  const int o_raw = 4 * orow + (lane >> 4);
  const bool live = o_raw < R && b0 < B;
  const int o = min(o_raw, R - 1);
  const int64_t b1 = min(b0 + nbi, B);
  const int64_t e0 = (int64_t)o * k;
  int ch[PER];
  float av[PER], wv[PER];
#pragma unroll
  for (int t = 0; t < PER; ++t) {
    const int i = min(h + 16 * t, k - 1);
    ch[t] = s[e0 + i];
    av[t] = a[e0 + i];
    wv[t] = w[e0 + i];
  }
  const float co = c[o];
  // descriptor gathers of image bb (clamped into the wave's range: the read
  // is issued on every pass, its value used only where bb is live)
  float dv[PER];
  auto gather = [&](int64_t bb, float (&v)[PER]) __attribute__((always_inline)) {
    const float* db = d + min(bb, B - 1) * C;
#pragma unroll
    for (int t = 0; t < PER; ++t) v[t] = db[ch[t]];
  };
  gather(b0, dv);
  for (int64_t b = b0; b < b1; ++b) {
    float dn[PER];
    gather(b + 1 < b1 ? b + 1 : b, dn);
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
    const int64_t item = b * R + o;
    if (live) {
      if (h == 0) tau[item] = tv;
      if (alpha) {
#pragma unroll
        for (int t = 0; t < PER; ++t)
          if (h + 16 * t < k) alpha[item * k + h + 16 * t] = coef_alpha(z[t], rzs);
      }
      if (st.rt && h == 0) put_stats(st, b, o, rt, m, rzs);
    }
#pragma unroll
    for (int t = 0; t < PER; ++t) dv[t] = dn[t];
  }
}

// The value of lane l ^ OFF within groups of 8 lanes (OFF = 1, 2, 4).
template <int OFF>
__device__ __forceinline__ float row8_xor(float v, int lane) {
  static_assert(OFF == 1 || OFF == 2 || OFF == 4, "within 8 lanes");
  return row16_xor<OFF>(v, lane);
}
__device__ __forceinline__ float row8_sum(float v, int lane) {
  v += row8_xor<4>(v, lane);
  v += row8_xor<2>(v, lane);
  v += row8_xor<1>(v, lane);
  return v;
}
__device__ __forceinline__ float row8_max(float v, int lane) {
  v = fmaxf(v, row8_xor<4>(v, lane));
  v = fmaxf(v, row8_xor<2>(v, lane));
  v = fmaxf(v, row8_xor<1>(v, lane));
  return v;
}

// The softplus-linear gate for 32 < k <= 8 PER with the descriptors in LDS.
// A group of 8 lanes per routed expert: lane h holds the support positions
// 8 VW t + VW h + q (q < VW), read as VW-wide vectors so that a read
// instruction covers whole cache lines of 8 experts' rows.  A workgroup of
// kLdsGateThreads lanes holds 32 experts and walks `nbi` consecutive images;
// each image's descriptor row is copied into LDS once (direct
// global-to-LDS copies, issued while the previous image is formed), so the
// support gathers are LDS reads.  Since 1/tau > 0 and rounding is
// monotonic, the largest scaled logit is the largest logit scaled:
// m = coef_z(max_i w_i, rt) has the bits of max_i coef_z(w_i, rt), and the
// maximum of the logits is taken once per expert instead of once per image.
constexpr int kLdsGateMaxC = 4096;  // descriptor rows of at most 16 KB
constexpr int kGateRing = 4;       // descriptor rows in LDS: the current one and two in flight
constexpr int kLdsGateThreads = 256;
constexpr int kLdsGateExperts = kLdsGateThreads / 8;

template <int VW>
struct VecOf;
template <>
struct VecOf<1> {
  using f = float;
  using i = int;
};
template <>
struct VecOf<2> {
  using f = float2;
  using i = int2;
};
template <>
struct VecOf<4> {
  using f = float4;
  using i = int4;
};
template <int VW, typename V>
__device__ __forceinline__ auto vget(const V& v, int q) {
  if constexpr (VW == 1) {
    return v;
  } else if constexpr (VW == 2) {
    return q == 0 ? v.x : v.y;
  } else {
    return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
  }
}

// waits until at most n (0 <= n <= 63) vector memory operations of this wave
// are outstanding (one s_waitcnt with a constant operand per possible n)
template <int... Ns>
__device__ __forceinline__ void wait_vm_of(int n, std::integer_sequence<int, Ns...>) {
  ((n == Ns ? (__builtin_amdgcn_s_waitcnt((Ns & 15) | ((Ns >> 4) << 14) | 0x0f70), 0) : 0), ...);
}
__device__ __forceinline__ void wait_vm_at_most(int n) { wait_vm_of(n, std::make_integer_sequence<int, 64>{}); }

template <int PER, int VW>
__global__ void __launch_bounds__(kLdsGateThreads)
k_gate_softplus_lds(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                    const float* __restrict__ a, const float* __restrict__ c, float* __restrict__ tau,
                    float* __restrict__ alpha, Stats st, int64_t B, int C, int R, int k, int nblk, int nbi) {
  static_assert(PER % VW == 0, "whole vectors");
  constexpr int NV = PER / VW;
  using VF = typename VecOf<VW>::f;
  using VI = typename VecOf<VW>::i;
  // LDS: kGateRing descriptor rows of cpad floats (C rounded up to 64), then
  // the results (tau, rt, m, rzs) of the workgroup's experts for each image
  extern __shared__ float gsm[];
  const int cpad = (C + 63) & ~63;
  float4* res = reinterpret_cast<float4*>(gsm + kGateRing * cpad);
  const int lane = threadIdx.x & 63;
  const int h = lane & 7;
  const int ex = threadIdx.x >> 3;  // expert slot within the workgroup
  const int64_t b0 = (int64_t)(blockIdx.x / nblk) * nbi;
  const int o0 = (blockIdx.x % nblk) * kLdsGateExperts;
  const int o = min(o0 + ex, R - 1);
  const int nimg = (int)(min(b0 + nbi, B) - b0);
  // position of element q of vector t of this lane (k need not fill the last
  // vectors; a vector that starts past k is read from the row's first
  // entries)
  auto pos = [&](int t, int q) __attribute__((always_inline)) { return 8 * VW * t + VW * h + q; };
  // descriptor row of image i (clamped into the workgroup's images) into
  // ring slot i % kGateRing by direct global-to-LDS copies.  Every wave
  // issues exactly fpw copies per row (64-float pieces v, v + nwaves, ...,
  // the last piece repeated where the row runs out; a piece past C repeats
  // entry C - 1 into the padding), so a row is complete once at most
  // fpw times the number of rows issued after it are outstanding.
  const int wv_id = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
  const int npieces = cpad / 64;
  const int fpw = (npieces + nwaves - 1) / nwaves;
  auto fetch = [&](int i) __attribute__((always_inline)) {
    const float* db = d + (b0 + min(i, nimg - 1)) * C;
    float* buf = gsm + (i % kGateRing) * cpad;
    for (int u = 0; u < fpw; ++u) {
      const int q = min(wv_id + nwaves * u, npieces - 1);
      __builtin_amdgcn_global_load_lds((const void*)(db + min(q * 64 + lane, C - 1)),
                                       (__attribute__((address_space(3))) void*)(buf + q * 64), 4, 0, 0);
    }
  };
  // the first rows go out before the expert rows' loads, so that both
  // arrive in one round trip
#pragma unroll
  for (int i = 0; i < kGateRing - 1; ++i) fetch(i);
  int ch[PER];
  float av[PER], wv[PER];
  float wmax = -INFINITY;
#pragma unroll
  for (int t = 0; t < NV; ++t) {
    const int64_t base = (int64_t)o * k + (pos(t, 0) < k ? pos(t, 0) : 0);
    const VI sv = *reinterpret_cast<const VI*>(s + base);
    const VF avv = *reinterpret_cast<const VF*>(a + base);
    const VF wvv = *reinterpret_cast<const VF*>(w + base);
#pragma unroll
    for (int q = 0; q < VW; ++q) {
      // a position past k adds nothing: gate weight 0 (at a valid channel)
      // and logit -inf (coefficient exp2(-inf) = 0), so no lane branches
      const bool in = pos(t, q) < k;
      ch[VW * t + q] = in ? vget<VW>(sv, q) : 0;
      av[VW * t + q] = in ? vget<VW>(avv, q) : 0.f;
      wv[VW * t + q] = in ? vget<VW>(wvv, q) : -INFINITY;
      wmax = fmaxf(wmax, wv[VW * t + q]);
    }
  }
  wmax = row8_max(wmax, lane);
  const float co = c[o];
  wait_vm_at_most((kGateRing - 2) * fpw);  // row 0 has landed
  __syncthreads();
  for (int i = 0; i < nimg; ++i) {
    // slot (i + kGateRing - 1) % kGateRing was last read for image i - 1,
    // before the barrier that ended it
    fetch(i + kGateRing - 1);
    const float* dr = gsm + (i % kGateRing) * cpad;
    float g = 0.f;
#pragma unroll
    for (int t = 0; t < PER; ++t) g += av[t] * dr[ch[t]];
    g = row8_sum(g, lane) + co;
    const float tv = softplusf(g) + 1e-3f;
    const float rt = 1.f / tv;
    const float m = coef_z(wmax, rt);
    float zs = 0.f;
    float z[PER];
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      z[t] = coef_e(coef_z(wv[t], rt), m);
      zs += z[t];
    }
    zs = row8_sum(zs, lane);
    const float rzs = 1.f / zs;
    if (h == 0) res[i * kLdsGateExperts + ex] = make_float4(tv, rt, m, rzs);
    if (alpha && o0 + ex < R) {
      const int64_t item = (b0 + i) * R + o;
#pragma unroll
      for (int t = 0; t < NV; ++t)
#pragma unroll
        for (int q = 0; q < VW; ++q)
          if (pos(t, q) < k) alpha[item * k + pos(t, q)] = coef_alpha(z[VW * t + q], rzs);
    }
    wait_vm_at_most((kGateRing - 2) * fpw);  // row i + 1 has landed
    __syncthreads();
  }
  // the results, image by image, 32 consecutive experts each
  for (int idx = threadIdx.x; idx < nimg * kLdsGateExperts; idx += blockDim.x) {
    const int i = idx / kLdsGateExperts, e = idx - i * kLdsGateExperts;
    if (o0 + e >= R) continue;
    const int64_t item = (b0 + i) * R + o0 + e;
    const float4 r4 = res[idx];
    tau[item] = r4.x;
    if (st.rt) put_stats(st, b0 + i, o0 + e, r4.y, r4.z, r4.w);
  }
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
  softmax_epilogue(w + (int64_t)o * k, k, t, lane, alpha ? alpha + item * k : nullptr, st.rt ? &st : nullptr, b,
                   o);
}

// The paper's gate as a batched product on the matrix cores, for k <= 128:
// H = ReLU(Z W1^T + b1) over the rows Z = d(b)[S'_o] of a block of 128
// experts of one image, then g = H w2 + b2 and tau as above.  Z and W1 are
// float32, split exactly into three bf16 parts each (hi + mid + lo, see
// split3_pair); the
// product keeps the six part products whose order is at most 2^-16 (hi hi,
// hi mid, mid hi, hi lo, mid mid, lo hi), accumulated in float32 by
// v_mfma_f32_16x16x32_bf16.  k is padded to KP (a multiple of 32) with zero
// inputs, zero weights and zero w2 entries, which add nothing.  W1's parts
// are staged in LDS once per workgroup, in rows of KP bf16 whose 16-byte
// chunks are rotated so that the 16 rows one B-fragment read touches fall in
// distinct bank groups; the workgroup then walks `nbi` images, restaging only
// the image's descriptor row.  The softmax statistics follow with a group of
// 8 lanes per expert, as in the softplus gate above.
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 gbf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float gf32x4;
typedef unsigned int gu32x4 __attribute__((ext_vector_type(4)));
constexpr int kMlpRows = 128;  // experts of one image per workgroup: 4 waves x 32
constexpr int kMlpMaxK = 128;
constexpr size_t kMlpMaxLds = 160 * 1024;  // per CU
constexpr int kMlpRowRegs = 16;           // descriptor entries per thread: C < 16 x 256
constexpr int64_t kMlpTargetBlocks = 256;

int mlp_kp(int k) { return k <= 32 ? 32 : k <= 64 ? 64 : 128; }
size_t mlp_lds_bytes(const Shape& sh) {
  const size_t kp = (size_t)mlp_kp(sh.k);
  return 3 * kp * kp * 2 + (size_t)kMlpRows * kp * 2 + (2 * kp + kMlpRows + 2 * ((size_t)sh.C + 1)) * sizeof(float);
}

// Two floats split exactly into three bf16 parts each, by truncation: the
// top 16 bits of a float are a bf16 value (8 significant bits); the
// remainder is exact and holds at most 16 significant bits, whose top 8 are
// the second part and whose last 8 are the third, each exact in bf16.  The
// parts come packed in pairs (first float low), one v_perm per pair.
__device__ __forceinline__ void split3_pair(float f0, float f1, uint32_t& p0, uint32_t& p1, uint32_t& p2) {
#pragma clang fp contract(off)
  constexpr uint32_t kHi = 0xffff0000u, kSel = 0x07060302u;  // the high halves of (src1, src0)
  const uint32_t u0 = __float_as_uint(f0), u1 = __float_as_uint(f1);
  p0 = __builtin_amdgcn_perm(u1, u0, kSel);
  const float r0 = f0 - __uint_as_float(u0 & kHi), r1 = f1 - __uint_as_float(u1 & kHi);
  const uint32_t v0 = __float_as_uint(r0), v1 = __float_as_uint(r1);
  p1 = __builtin_amdgcn_perm(v1, v0, kSel);
  const float q0 = r0 - __uint_as_float(v0 & kHi), q1 = r1 - __uint_as_float(v1 & kHi);
  p2 = __builtin_amdgcn_perm(__float_as_uint(q1), __float_as_uint(q0), kSel);
}

template <int KP>
__global__ void __launch_bounds__(kGateWaves * kWave)
k_gate_mlp_mfma(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ w,
                const float* __restrict__ W1, const float* __restrict__ b1, const float* __restrict__ w2, float b2,
                float tau_min, float tau_max, float* __restrict__ tau, float* __restrict__ alpha, Stats st,
                int64_t B, int C, int R, int k, int nblk, int nbi) {
  static_assert(KP % 32 == 0 && KP <= kMlpMaxK, "K padded to whole 32-deep slices");
  constexpr int kChunks = KP / 8;                       // 16-byte chunks of a W1 row
  constexpr int kSh = KP == 128 ? 0 : KP == 64 ? 1 : 2;  // rows sharing a 256-byte bank span
  constexpr int kPer = KP / 8;                          // logits per lane in the softmax (8 lanes an expert)
  // LDS: W1's parts [3][KP][KP] bf16, the block's supports [kMlpRows][KP] as
  // 16-bit channels (C marks a padding position), b1 and w2 [KP], the
  // temperatures [kMlpRows], then the image's descriptor row [C + 1] whose
  // entry C is 0
  extern __shared__ float gsm[];
  uint16_t* wl = reinterpret_cast<uint16_t*>(gsm);
  uint16_t* sl16 = wl + 3 * KP * KP;
  float* b1s = reinterpret_cast<float*>(sl16 + kMlpRows * KP);
  float* w2s = b1s + KP;
  float* taus = w2s + KP;
  float* dr = taus + kMlpRows;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int n = lane & 15, gq = lane >> 4;
  const int64_t b0 = (int64_t)(blockIdx.x / nblk) * nbi;
  const int o0 = (blockIdx.x % nblk) * kMlpRows;
  const int64_t b1e = min(b0 + nbi, B);
  // element (j, i) of a part: chunk i / 8 of row j stored at chunk
  // (i / 8) ^ ((j >> kSh) & (kChunks - 1))
  auto wl_at = [&](int part, int j, int chunk) __attribute__((always_inline)) {
    return wl + (part * KP + j) * KP + ((chunk ^ ((j >> kSh) & (kChunks - 1))) << 3);
  };
  // W1 by 8-wide chunks: every thread first reads all of its chunks, then
  // splits and stores them
  constexpr int kW1Per = (KP * kChunks + kGateWaves * kWave - 1) / (kGateWaves * kWave);
  float wv8[kW1Per][8];
#pragma unroll
  for (int u = 0; u < kW1Per; ++u) {
    const int idx = threadIdx.x + kGateWaves * kWave * u;
    const int j = idx / kChunks, c8 = idx - j * kChunks;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = 8 * c8 + q;
      // read unconditionally (clamped into W1) and then selected: a read
      // under a lane condition would be waited for on its own
      const float v = W1[(int64_t)min(j, k - 1) * k + min(i, k - 1)];
      wv8[u][q] = idx < KP * kChunks && j < k && i < k ? v : 0.f;
    }
  }
#pragma unroll
  for (int u = 0; u < kW1Per; ++u) {
    const int idx = threadIdx.x + kGateWaves * kWave * u;
    if (idx >= KP * kChunks) continue;
    const int j = idx / kChunks, c8 = idx - j * kChunks;
    gu32x4 v0, v1, v2;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      uint32_t q0, q1, q2;
      split3_pair(wv8[u][2 * h], wv8[u][2 * h + 1], q0, q1, q2);
      v0[h] = q0;
      v1[h] = q1;
      v2[h] = q2;
    }
    *reinterpret_cast<gu32x4*>(wl_at(0, j, c8)) = v0;
    *reinterpret_cast<gu32x4*>(wl_at(1, j, c8)) = v1;
    *reinterpret_cast<gu32x4*>(wl_at(2, j, c8)) = v2;
  }
  // the block's supports, as 16-bit channels; padding positions and rows
  // past R point at the zero entry C
  // (all of a thread's reads issued before any is used)
  constexpr int kSPer = kMlpRows * KP / (kGateWaves * kWave);
  int32_t sv[kSPer];
#pragma unroll
  for (int u = 0; u < kSPer; ++u) {
    const int idx = threadIdx.x + kGateWaves * kWave * u;
    const int r = idx / KP, i = idx - r * KP;
    sv[u] = s[(int64_t)min(o0 + r, R - 1) * k + min(i, k - 1)];
  }
#pragma unroll
  for (int u = 0; u < kSPer; ++u) {
    const int idx = threadIdx.x + kGateWaves * kWave * u;
    const int r = idx / KP, i = idx - r * KP;
    sl16[idx] = (uint16_t)(o0 + r < R && i < k ? sv[u] : C);
  }
  for (int j = threadIdx.x; j < KP; j += blockDim.x) {
    const float v1 = b1[min(j, k - 1)], v2 = w2[min(j, k - 1)];
    b1s[j] = j < k ? v1 : 0.f;
    w2s[j] = j < k ? v2 : 0.f;
  }
  // this wave's 32 rows: blocks mb = 0, 1 of 16; lane (gq, n) builds the A
  // fragment of row 32 wv + 16 mb + n, supports 32 sl + 8 gq .. + 7
  // the logits of the wave's 32 experts for the softmax (8 lanes an
  // expert, 8 experts a pass, 4 passes), held across the images with
  // their maxima
  const int h8 = lane & 7;
  float wr[4][kPer], wmx[4];
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int o = min(o0 + 32 * wv + 8 * pass + (lane >> 3), R - 1);
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int i = h8 + 8 * t;
      const float v = w[(int64_t)o * k + min(i, k - 1)];
      wr[pass][t] = i < k ? v : -INFINITY;
      mx = fmaxf(mx, wr[pass][t]);
    }
    wmx[pass] = row8_max(mx, lane);
  }
  // descriptor rows in two buffers of C + 1 floats (entry C is 0): image
  // b + 1's row is read into registers while image b is formed
  {
    float v[kMlpRowRegs];
#pragma unroll
    for (int u = 0; u < kMlpRowRegs; ++u) v[u] = d[b0 * C + min((int)threadIdx.x + kGateWaves * kWave * u, C - 1)];
#pragma unroll
    for (int u = 0; u < kMlpRowRegs; ++u) {
      const int c = threadIdx.x + kGateWaves * kWave * u;
      if (c <= C) dr[c] = c < C ? v[u] : 0.f;
    }
  }
  for (int64_t b = b0; b < b1e; ++b) {
    const int cur = (int)((b - b0) & 1);
    const float* drc = dr + cur * (C + 1);  // this image's row (LDS, indexed from the shared base)
    __syncthreads();  // this image's row is in place; the previous image's reads of taus are done
    float nxt[kMlpRowRegs];
    const int64_t bn = b + 1 < b1e ? b + 1 : b;
#pragma unroll
    for (int u = 0; u < kMlpRowRegs; ++u) {
      const int c = threadIdx.x + kGateWaves * kWave * u;
      const float v = d[bn * C + min(c, C - 1)];
      nxt[u] = c < C ? v : 0.f;
    }
    gf32x4 acc[2][KP / 16];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < KP / 16; ++nb) acc[mb][nb] = gf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sl = 0; sl < KP / 32; ++sl) {
      gbf16x8 a[2][3];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const gu32x4 c8 =
            *reinterpret_cast<const gu32x4*>(sl16 + (32 * wv + 16 * mb + n) * KP + 32 * sl + 8 * gq);
        gu32x4 v0, v1, v2;
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          uint32_t q0, q1, q2;
          split3_pair(drc[c8[h] & 0xffff], drc[c8[h] >> 16], q0, q1, q2);
          v0[h] = q0;
          v1[h] = q1;
          v2[h] = q2;
        }
        a[mb][0] = __builtin_bit_cast(gbf16x8, v0);
        a[mb][1] = __builtin_bit_cast(gbf16x8, v1);
        a[mb][2] = __builtin_bit_cast(gbf16x8, v2);
      }
      // every B fragment of the slice first, then the six part products
      // each over all 2 KP / 16 accumulators, so that consecutive products
      // into one accumulator are that many MFMAs apart
      gbf16x8 bf[KP / 16][3];
#pragma unroll
      for (int nb = 0; nb < KP / 16; ++nb)
#pragma unroll
        for (int pt = 0; pt < 3; ++pt)
          bf[nb][pt] =
              __builtin_bit_cast(gbf16x8, *reinterpret_cast<const gu32x4*>(wl_at(pt, 16 * nb + n, 4 * sl + gq)));
      constexpr int kPa[6] = {2, 1, 0, 1, 0, 0}, kPb[6] = {0, 1, 2, 0, 1, 0};  // smallest terms first
#pragma unroll
      for (int t = 0; t < 6; ++t)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int nb = 0; nb < KP / 16; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mb][kPa[t]], bf[nb][kPb[t]], acc[mb][nb], 0, 0, 0);
    }
    // lane (gq, n) holds H[16 mb + 4 gq + r][16 nb + n]: bias, ReLU, w2 and
    // the sum over the hidden units (its 16 lanes hold the 16 columns)
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float gp = 0.f;
#pragma unroll
        for (int nb = 0; nb < KP / 16; ++nb)
          gp += fmaxf(acc[mb][nb][r] + b1s[16 * nb + n], 0.f) * w2s[16 * nb + n];
        gp = row16_sum(gp, lane) + b2;
        if (n == 0) taus[32 * wv + 16 * mb + 4 * gq + r] = tau_min + (tau_max - tau_min) / (1.f + expf(-gp));
      }
    __syncthreads();
    // softmax over each expert's logits
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int row = 32 * wv + 8 * pass + (lane >> 3);
      const int o_raw = o0 + row;
      const int o = min(o_raw, R - 1);
      const float tv = taus[row];
      const float rt = 1.f / tv;
      const float m = coef_z(wmx[pass], rt);
      float z[kPer];
      float zs = 0.f;
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        z[t] = coef_e(coef_z(wr[pass][t], rt), m);
        zs += z[t];
      }
      zs = row8_sum(zs, lane);
      const float rzs = 1.f / zs;
      if (o_raw < R) {
        const int64_t item = b * R + o;
        if (h8 == 0) tau[item] = tv;
        if (alpha) {
#pragma unroll
          for (int t = 0; t < kPer; ++t)
            if (h8 + 8 * t < k) alpha[item * k + h8 + 8 * t] = coef_alpha(z[t], rzs);
        }
        if (st.rt && h8 == 0) put_stats(st, b, o, rt, m, rzs);
      }
    }
    // the next image's row into the other buffer (last read two images ago)
    if (b + 1 < b1e) {
      float* dn = dr + (1 - cur) * (C + 1);
#pragma unroll
      for (int u = 0; u < kMlpRowRegs; ++u) {
        const int c = threadIdx.x + kGateWaves * kWave * u;
        if (c <= C) dn[c] = nxt[u];
      }
    }
  }
}

}  // namespace

hipError_t launch_gate(const Shape& sh, const float* d, const int32_t* s, const float* w,
                       const moce_gate_params& g, float* tau, float* alpha, float* stats, hipStream_t st) {
  if (sh.R == 0) return hipSuccess;
  const int64_t items = sh.B * sh.R;
  const Stats sp = stats ? stats_planes(stats, items, sh.R, 1) : Stats{nullptr, nullptr, nullptr, 0, 0};
  const unsigned blocks = (unsigned)((items + kGateWaves - 1) / kGateWaves);
  if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 32) {
    // segments of 8, 16 or 32 lanes: the narrowest that holds k (the sums and
    // maxima over the lanes past k add zeros, so every width gives the same
    // bits)
    const int W = sh.k <= 8 ? 8 : sh.k <= 16 ? 16 : 32;
    const int64_t per = (int64_t)kGateWaves * (kWave / W);
    const unsigned bs = (unsigned)((items + per - 1) / per);
    using K = void (*)(const float*, const int32_t*, const float*, const float*, const float*, float*, float*, Stats,
                       int64_t, int64_t, int, int);
    const K kf = W == 8 ? k_gate_softplus_seg<8> : W == 16 ? k_gate_softplus_seg<16> : k_gate_softplus_seg<32>;
    hipLaunchKernelGGL(kf, dim3(bs), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c, tau, alpha, sp, sh.B,
                       sh.C, sh.R, sh.k);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 128 && sh.C <= kLdsGateMaxC) {
    // 32 experts per workgroup, nbi images each, for about kLdsGateTargetBlocks
    // workgroups
    const int nblk = (int)((sh.R + kLdsGateExperts - 1) / kLdsGateExperts);
    const int64_t nbi = std::min<int64_t>(
        kLdsGateMaxImages, std::max<int64_t>(1, ((int64_t)nblk * sh.B + kLdsGateTargetBlocks - 1) / kLdsGateTargetBlocks));
    const unsigned grid = (unsigned)(nblk * ((sh.B + nbi - 1) / nbi));
    const size_t lds = (kGateRing * ((sh.C + 63) / 64 * 64) + nbi * kLdsGateExperts * 4) * sizeof(float);
    const int per = (sh.k + 7) / 8;
    // vectors of 4 (or 2) positions where k fills whole rounds of them and
    // the three arrays are aligned to the vector
    auto aligned = [&](size_t bytes) {
      return ((reinterpret_cast<uintptr_t>(s) | reinterpret_cast<uintptr_t>(g.a) | reinterpret_cast<uintptr_t>(w)) &
              (bytes - 1)) == 0;
    };
    const int vw = sh.k % 32 == 0 && aligned(16) ? 4 : sh.k % 16 == 0 && aligned(8) ? 2 : 1;
    using K = void (*)(const float*, const int32_t*, const float*, const float*, const float*, float*, float*, Stats,
                       int64_t, int, int, int, int, int);
    K kern = per <= 4 ? (vw == 4 ? k_gate_softplus_lds<4, 4> : vw == 2 ? k_gate_softplus_lds<4, 2> : k_gate_softplus_lds<4, 1>)
             : per <= 6 ? (vw == 2 ? k_gate_softplus_lds<6, 2> : k_gate_softplus_lds<6, 1>)
             : per <= 8 ? (vw == 4 ? k_gate_softplus_lds<8, 4> : vw == 2 ? k_gate_softplus_lds<8, 2> : k_gate_softplus_lds<8, 1>)
                        : (vw == 4 ? k_gate_softplus_lds<16, 4> : vw == 2 ? k_gate_softplus_lds<16, 2> : k_gate_softplus_lds<16, 1>);
    if (lds > 64 * 1024) {
      const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kLdsGateThreads), lds, st, d, s, w, g.a, g.c, tau, alpha, sp, sh.B,
                       (int)sh.C, sh.R, sh.k, nblk, (int)nbi);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k <= 256) {
    // rows of 16 lanes, four experts per wave; each wave walks nbi images,
    // nbi chosen for about 16 waves per CU
    const int nrow = (int)((sh.R + 3) / 4);
    const int64_t nbi = std::max<int64_t>(1, ((int64_t)nrow * sh.B + kGateTargetWaves - 1) / kGateTargetWaves);
    const int64_t waves = (int64_t)nrow * ((sh.B + nbi - 1) / nbi);
    const unsigned b16 = (unsigned)((waves + kGateWaves - 1) / kGateWaves);
    const int per = (sh.k + 15) / 16;
    auto kern = per <= 4 ? k_gate_softplus_x16<4> : per <= 8 ? k_gate_softplus_x16<8> : k_gate_softplus_x16<16>;
    hipLaunchKernelGGL(kern, dim3(b16), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c, tau, alpha, sp, sh.B,
                       sh.C, sh.R, sh.k, nrow, (int)nbi);
  } else if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR) {
    hipLaunchKernelGGL(k_gate_softplus, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.a, g.c,
                       tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  } else if (sh.k <= kMlpMaxK && mlp_lds_bytes(sh) <= kMlpMaxLds && sh.C < kMlpRowRegs * kGateWaves * kWave) {
    // the batched product: 128 experts of an image per workgroup, nbi images
    // each (W1 and the supports staged once), for about one workgroup per CU
    const int nblk = (int)((sh.R + kMlpRows - 1) / kMlpRows);
    const int64_t nbi = std::max<int64_t>(1, ((int64_t)nblk * sh.B + kMlpTargetBlocks - 1) / kMlpTargetBlocks);
    const unsigned grid = (unsigned)(nblk * ((sh.B + nbi - 1) / nbi));
    const int kp = mlp_kp(sh.k);
    const size_t lds = mlp_lds_bytes(sh);
    using K = void (*)(const float*, const int32_t*, const float*, const float*, const float*, const float*, float,
                       float, float, float*, float*, Stats, int64_t, int, int, int, int, int);
    const K kern = kp == 32 ? k_gate_mlp_mfma<32> : kp == 64 ? k_gate_mlp_mfma<64> : k_gate_mlp_mfma<128>;
    if (lds > 64 * 1024) {
      const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kGateWaves * kWave), lds, st, d, s, w, g.W1, g.b1, g.w2, g.b2,
                       g.tau_min, g.tau_max, tau, alpha, sp, sh.B, (int)sh.C, sh.R, sh.k, nblk, (int)nbi);
  } else {
    hipLaunchKernelGGL(k_gate_mlp, dim3(blocks), dim3(kGateWaves * kWave), 0, st, d, s, w, g.W1, g.b1, g.w2,
                       g.b2, g.tau_min, g.tau_max, tau, alpha, sp, sh.B, sh.C, sh.R, sh.k);
  }
  return hipGetLastError();
}

}  // namespace moce

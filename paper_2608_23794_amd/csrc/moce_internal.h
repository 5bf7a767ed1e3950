// Internal declarations shared by the HIP translation units of libmoce.
// Device helpers for bfloat16 handling and wave64 reductions, plus the
// launchers that the C ABI layer (api.hip) dispatches to.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/moce.h"

namespace moce {

constexpr int kWave = 64;

// ---- bfloat16 <-> float32 ------------------------------------------------
// bf16 values travel as their 16-bit patterns (uint16_t).  Widening is exact:
// the pattern becomes the upper half of a float32.
__device__ __forceinline__ float bf16_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t pair) { return __uint_as_float(pair & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// float32 -> bf16, round to nearest even (the hardware conversion on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// ---- wave64 reductions ---------------------------------------------------
template <int WIDTH = kWave>
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = WIDTH / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, WIDTH);
  return v;
}
template <int WIDTH = kWave>
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = WIDTH / 2; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, WIDTH));
  return v;
}
__device__ __forceinline__ int wave_min_int(int v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, kWave));
  return v;
}

// softplus(t) = log(1 + e^t) = max(t, 0) + log1p(e), e = e^-|t| in (0, 1],
// from the hardware base-2 exponential and logarithm.  The rounding error of
// the exponential's argument -|t| log2(e) is fed back to first order (one
// FMA); log1p(e) is log(u) e / (u - 1) with u = 1 + e rounded, which cancels
// the rounding of u (and is e itself where u rounds to 1).  A few ulp over
// the whole range (relative error below 1e-6), in about 15 instructions
// where the library's log1pf(expf(.)) takes over a hundred.
__device__ __forceinline__ float softplusf(float t) {
#pragma clang fp contract(off)
  constexpr float kL2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  const float na = -fabsf(t);
  const float x = na * kL2e;
  const float dx = __builtin_fmaf(na, kL2e, -x);  // na log2(e) - x, exactly
  float e = __builtin_amdgcn_exp2f(x);
  e = __builtin_fmaf(e * kLn2, dx, e);            // e 2^dx to first order
  const float u = 1.f + e;
  const float l = u == 1.f ? e : (__builtin_amdgcn_logf(u) * kLn2) * (e * __builtin_amdgcn_rcpf(u - 1.f));
  return fmaxf(t, 0.f) + l;
}

// ---- mixing coefficients (Sec. 3.3 Eq. 4) ----------------------------------
// Every kernel forms coefficient i of routed expert o for image b with the
// same operations, so a coefficient that a mix kernel rebuilds from the
// softmax statistics of (b, o) equals the one a gate kernel writes, bit for
// bit:
//   rt = 1 / tau (IEEE division, once per (b, o)),   z_i = w_i * rt,
//   m = max_i z_i,   e_i = 2^((z_i - m) * log2(e)),  rzs = 1 / sum_i e_i,
//   alpha_i = e_i * rzs.
// The largest entry has z_i - m = 0 and e_i = 1 exactly, so k = 1 and the
// one-hot limit (tau -> 0 with a clear top logit) give coefficients of
// exactly 1.  The products and the difference are kept apart (no fused
// multiply-add), so the same bits come out wherever the helpers are inlined.
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float coef_z(float w, float rt) {
#pragma clang fp contract(off)
  return w * rt;
}
__device__ __forceinline__ float coef_e(float z, float m) {
#pragma clang fp contract(off)
  const float t = (z - m) * kLog2e;
  return __builtin_amdgcn_exp2f(t);
}
__device__ __forceinline__ float coef_alpha(float e, float rzs) {
#pragma clang fp contract(off)
  return e * rzs;
}

// Softmax statistics of the B*R (image, expert) pairs, three planes of n =
// B*R floats: rt[n], m[n], rzs[n]; pair (b, o) at b sb + o so, so image-major
// [B][R] (sb = R, so = 1) or expert-major [R][B] (sb = 1, so = B).
struct Stats {
  float* rt;
  float* m;
  float* rzs;
  int64_t sb, so;
};
__host__ __device__ inline Stats stats_planes(float* base, int64_t n, int64_t sb, int64_t so) {
  return Stats{base, base + n, base + 2 * n, sb, so};
}

// ---- output epilogue -------------------------------------------------------
// y[.][o][.] = act(scale[o] v + shift[o]) applied to a float32 output value v
// before it is rounded and stored: a per-output-channel affine map (a folded
// inference batch norm) and an optional ReLU.  scale == nullptr: no affine
// map.
struct Epi {
  const float* scale;
  const float* shift;
  int relu;
};
__device__ __forceinline__ float epi_apply(const Epi& e, float v, int o) {
  if (e.scale) v = __builtin_fmaf(v, e.scale[o], e.shift[o]);
  if (e.relu) v = fmaxf(v, 0.f);
  return v;
}
__host__ __device__ inline bool epi_active(const Epi& e) { return e.scale != nullptr || e.relu != 0; }

// ---- launch parameters derived from a validated descriptor ---------------
struct Shape {
  int64_t B, C, HW;
  int E, R, k;       // R = E - 1 routed experts
  int elem;          // MOCE_F32 / MOCE_BF16
  int layout;        // MOCE_NCHW / MOCE_NHWC
};

// ---- launchers (return hipSuccess or the launch error) --------------------
// s: int32 channel indices, or uint16 ones when s16 (the 16-bit storage of
// deployed supports)
hipError_t launch_prepare(const Shape& sh, const void* s, bool s16, const float* w, int32_t* s_out,
                          float* w_out, uint8_t* covered, int32_t* U, int32_t* info,
                          hipStream_t st);
hipError_t launch_pool(const Shape& sh, const void* x, float* d, hipStream_t st);
// tau [B][R] is always written; alpha and the softmax statistics (a block of
// 3 B R floats, image-major planes as in stats_planes) are optional outputs
// (nullptr: not written).
hipError_t launch_gate(const Shape& sh, const float* d, const int32_t* s, const float* w,
                       const moce_gate_params& g, float* tau, float* alpha, float* stats, hipStream_t st);

// alpha != nullptr: coefficients are read from alpha[B][R][k]; otherwise
// they are rebuilt from the logits w and the softmax statistics (a block of
// 3 B R floats), with the gate's operations.
hipError_t launch_mix(const Shape& sh, const void* x, const int32_t* s, const float* alpha,
                      const float* w, const float* stats, const int32_t* U, int nU,
                      void* y, hipStream_t st);

// Tile gather-mix for NCHW bfloat16 with C <= 256 (tilemix.hip), from the
// coefficients alpha [B][R][k].
bool tilemix_eligible(const Shape& sh);
size_t tilemix_lds_bytes(const Shape& sh);
hipError_t launch_tilemix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st);
// The same mix with input-conditioned supports S [B][R][k], uncovered lists
// U [B][C] and counts nU [B].
bool tilemix_dynamic_eligible(const Shape& sh);
hipError_t launch_tilemix_dynamic(const Shape& sh, const void* x, const int32_t* S, const float* alpha,
                                  const int32_t* U, const int32_t* nU, void* y, hipStream_t st);

// Mixing as a dense bf16 product on the matrix cores (mfmamix.hip), for NCHW
// bfloat16 with R >= 1, C a multiple of 32 up to 256, E <= 64 and H*W a
// multiple of 8; supports must hold distinct channels (prepared rows).
bool mfmamix_eligible(const Shape& sh);
hipError_t launch_mfmamix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st,
                   const Epi& ep = Epi{});
// The same product with the softplus-linear gate evaluated inside the mix
// kernel from the pooled descriptors d (bit-identical coefficients, no
// temperatures or coefficients written), for k = 32.
bool mfmamix_gate_fusable(const Shape& sh, int gate_kind);
hipError_t launch_mfmamix_gated(const Shape& sh, const void* x, const int32_t* s, const float* w, const float* d,
                                const float* a, const float* c, const int32_t* U, int nU, void* y, hipStream_t st,
                   const Epi& ep = Epi{});

// Channels-last bfloat16 mixing on the matrix cores from a per-forward
// channel schedule of the supports (gmix.hip): C a multiple of 64 up to 4096,
// E a multiple of 8.  launch_pool_sched pools x into d and builds the
// schedule (gmix_sched_bytes(sh) of device workspace) in one launch;
// launch_gmix then mixes, rebuilding the coefficients from the softmax
// statistics (a block of 3 B R floats written by launch_gate).
bool gmix_eligible(const Shape& sh);
size_t gmix_sched_bytes(const Shape& sh);
hipError_t launch_pool_sched(const Shape& sh, const void* x, float* d, const int32_t* s, const float* w,
                             const int32_t* U, int nU, void* sched, hipStream_t st);
// Channels-last bfloat16 gather mixing for small supports (gather.hip): k <=
// 16, C a multiple of 8 up to 4096, E-1 <= 1024 (512 for k > 8); coefficients from alpha
// [B][R][k], the epilogue applied before rounding.
bool gather_eligible(const Shape& sh);
hipError_t launch_gather(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                         int nU, void* y, hipStream_t st, const Epi& ep);

// The epilogue applied in place to a finished y (the paths whose mix kernels
// do not apply it themselves).
hipError_t launch_epilogue(const Shape& sh, void* y, const Epi& ep, hipStream_t st);
hipError_t launch_gmix(const Shape& sh, const void* x, const float* stats, int nU, const void* sched, void* y,
                       hipStream_t st,
                   const Epi& ep = Epi{});

// Input-conditioned supports (dynamic.hip): the whole inference path from x
// to y over workspace arrays: the router output h [B][d], the transposed
// channel embeddings vT [d][C], per-example supports S [B][R][k] and their
// logits W, per-example
// uncovered sets U [B][C] with counts nU [B], temperatures and coefficients,
// over the workspace arrays passed in.
bool dynamic_supported(const Shape& sh, int d);
hipError_t launch_dynamic(const Shape& sh, const void* x, const float* L, const moce_router& r,
                          const moce_gate_params& g, void* y, float* d, float* h, float* vT, int32_t* S, float* W,
                          int32_t* U, int32_t* nU, float* tau, float* alpha, hipStream_t st);

// Backward (backward.hip, bwdmfma.hip).  Device arrays of the workspace:
// d [B][C], tau [B][R], stats [3][B][R] (image-major planes), alpha, dal [B][R][k],
// S1, dtau, dg [B][R], dd [B][C], the inverse support map (cnt, cur [C],
// off [C+1], inv [R k], nU [1]), and for the MLP gate dzg [B][R][k] and
// part (the per-workgroup partial sums).
struct BwdWs {
  float* d;
  float* tau;
  float* stats;
  float* alpha;
  float* dal;
  float* S1;
  float* dtau;
  float* dg;
  float* dd;
  int32_t* cnt;
  int32_t* cur;
  int32_t* off;
  int32_t* inv;
  int32_t* nU;
  float* dzg;
  float* part;
  // the matrix-core dx: bucket counts, offsets [nb + 1] and cursors, the
  // scheduled entries (w0, w1) and their coefficients per image [B][NEmax]
  int32_t* dxs_cnt;
  int32_t* dxs_off;
  int32_t* dxs_cur;
  uint32_t* dxs_w0;
  int32_t* dxs_w1;
  uint32_t* dxs_coef;
  // partial sums over image groups: dw, da [ng][R k], dc [ng][R]
  float* psum;
};
void backward_sum_groups(const Shape& sh, int* ng, int* gs);
bool backward_supported(const Shape& sh, int gate_kind);
size_t backward_mlp_parts(const Shape& sh);
size_t backward_mlp_part_floats(const Shape& sh);
hipError_t launch_backward(const Shape& sh, const void* x, const void* dy, const int32_t* s, const float* w,
                           const moce_gate_params& g, void* dx, float* dw, const moce_gate_grads& gg,
                           const BwdWs& ws, hipStream_t st);
// The matrix-core kernels of the backward: each returns false (and launches
// nothing) where the shape does not suit it, else true with the launch status
// in *err.
bool bwd_mfma_dalpha(const Shape& sh, const void* x, const void* dy, const int32_t* s, const BwdWs& ws,
                     hipStream_t st, hipError_t* err);
// Partial sums of dalpha along the positions: dal holds nsplit blocks of
// B R k floats (nsplit = 1 except for the matrix-core NCHW product).
void bwd_dalpha_splits(const Shape& sh, int* nsplit, int* split_len);
bool bwd_mfma_dx(const Shape& sh, const void* dy, const int32_t* s, const float* w, const BwdWs& ws, void* dx,
                 hipStream_t st, hipError_t* err);
// sizes of the dx schedule (0 where the matrix-core dx does not apply)
void bwd_dx_sched_sizes(const Shape& sh, int* nbuckets, int64_t* ne_max);

// Coverage loss and the full routing-logit gradient; ws holds 2 R + C + 3 floats.
bool logit_backward_supported(int64_t C);
hipError_t launch_logit_backward(int R, int C, int k, const float* L, const int32_t* s, const float* dw, float eps,
                                 float lambda, float* loss, float* dL, float* ws, hipStream_t st);

}  // namespace moce

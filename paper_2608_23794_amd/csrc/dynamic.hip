// Input-conditioned supports (Sec. 4.5, Eq. 11), the inference path.
//
// The variant keeps the temperature gate and the residual, and replaces the
// static supports by per-example ones: a router reads the whole pooled
// descriptor z, h = ReLU(Wh z + bh) (d outputs), and adds a rank-d offset to
// the routing logits, L(X)[e][c] = L[e][c] + <q_e * h, v_c>.  Each example then
// takes its own top-k channels per routed expert, the gate reads z at that
// support, the coefficients are the softmax of L(X) at the support over the
// temperature, and the residual averages the channels in no support of that
// example.
//
// Launches: pooling (pool.hip), the router (a wave per (image, bottleneck
// unit)), selection (a workgroup per (image, block of EB experts): the block's
// logit rows are formed in LDS and each wave takes a row's top k by a radix
// select over order-preserving 32-bit keys, then sorts the k by (logit
// descending, channel ascending)), the per-example uncovered set (a workgroup
// per image), the gate and coefficients (a wave per (image, expert)), and the
// mix (a workgroup per (image, tile of positions) with the tile of every
// channel in LDS).
#include <algorithm>
#include <climits>
#include <initializer_list>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kDynThreads = 256;
constexpr int kDynWaves = kDynThreads / kWave;
constexpr size_t kDynLds = 160 * 1024;
constexpr int kDynMaxD = 64;     // bottleneck width
constexpr int kDynMaxC = 4096;   // the mix stages C channels x 8 positions of float

// ---------------------------------------------------------------- router
__global__ void __launch_bounds__(kDynThreads)
k_dyn_router(const float* __restrict__ d, const float* __restrict__ Wh, const float* __restrict__ bh,
             float* __restrict__ h, int64_t B, int C, int dd) {
  const int64_t wave = (int64_t)blockIdx.x * kDynWaves + (threadIdx.x >> 6);
  if (wave >= B * dd) return;  // whole waves
  const int lane = threadIdx.x & 63;
  const int64_t b = wave / dd;
  const int t = (int)(wave - b * dd);
  float acc = 0.f;
  for (int c = lane; c < C; c += kWave) acc += Wh[(int64_t)t * C + c] * d[b * C + c];
  acc = wave_sum(acc);
  if (lane == 0) h[wave] = fmaxf(acc + bh[t], 0.f);
}

// vT[t][c] = v[c][t]: the channel embeddings transposed, 32 x 32 tiles
// through LDS
__global__ void __launch_bounds__(1024)
k_dyn_transpose(const float* __restrict__ v, float* __restrict__ vT, int C, int dd) {
  __shared__ float tile[32][33];
  const int c0 = blockIdx.x * 32, t0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  if (c0 + ty < C && t0 + tx < dd) tile[ty][tx] = v[(int64_t)(c0 + ty) * dd + t0 + tx];
  __syncthreads();
  if (t0 + ty < dd && c0 + tx < C) vT[(int64_t)(t0 + ty) * C + c0 + tx] = tile[tx][ty];
}

// ---------------------------------------------------------------- selection
// Order-preserving key of a float (larger float, larger key); -0 is taken as
// +0 first, so that equal logits have equal keys.
__device__ __forceinline__ uint32_t fkey(float v) {
  const uint32_t u = __float_as_uint(v + 0.f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float fkey_value(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}
// (key a, channel a) comes before (key b, channel b): larger logit first,
// then the lower channel
__device__ __forceinline__ bool before(uint32_t ka, int ca, uint32_t kb, int cb) {
  return ka > kb || (ka == kb && ca < cb);
}
__device__ __forceinline__ void lds_wait() { __builtin_amdgcn_s_waitcnt(0xc07f); }  // lgkmcnt(0)

// LDS per wave for one row's selection: the radix histogram and the list of
// the selected (key, channel) pairs, kl = the power of two >= k entries
constexpr int kDynMaxK = 512;
__host__ __device__ inline int list_len(int k) {
  int P = 1;
  while (P < k) P <<= 1;
  return P;
}
__host__ __device__ inline int wave_words(int k) { return 256 + 2 * list_len(k); }

// The top k of one logit row by one wave: the k-th largest key by a radix
// select, most significant byte first, then the keys above it and the
// lowest-channel ones equal to it, sorted into the canonical order (logit
// descending, channel ascending).  hist: 256 words of LDS; lkey, lch: P
// entries each (P = list_len(k)), which may overlap hist.
__device__ __forceinline__ void select_row(const float* row, uint32_t* hist, uint32_t* lkey, int32_t* lch, int C,
                                           int k, int P, int lane, int32_t* __restrict__ Sout,
                                           float* __restrict__ Wout) {
    // the k-th largest key, most significant byte first: after each round,
  // `prefix` holds the known high bytes and kk the rank still to find
  // among the keys with that prefix
  uint32_t prefix = 0, mask = 0;
  int kk = k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = lane; i < 256; i += kWave) hist[i] = 0;
    lds_wait();
    for (int c = lane; c < C; c += kWave) {
      const uint32_t key = fkey(row[c]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    lds_wait();
    // lane l holds bins 4 l .. 4 l + 3; counts above a lane's bins by a
    // suffix sum over the lanes
    uint32_t cnt[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cnt[j] = hist[4 * lane + j];
    const uint32_t mine = cnt[0] + cnt[1] + cnt[2] + cnt[3];
    uint32_t incl = mine;  // sum over lanes >= this one
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint32_t o = __shfl_down(incl, off, kWave);
      if (lane + off < kWave) incl += o;
    }
    uint32_t above = incl - mine;
    int digit = -1;
    uint32_t before_digit = 0;
    if (above < (uint32_t)kk && (uint32_t)kk <= incl) {
#pragma unroll
      for (int j = 3; j >= 0; --j) {
        if (digit < 0 && above + cnt[j] >= (uint32_t)kk) {
          digit = 4 * lane + j;
          before_digit = above;
        }
        above += cnt[j];
      }
    }
    const uint64_t found = __ballot(digit >= 0);
    const int src = __builtin_ctzll(found);
    digit = __shfl(digit, src, kWave);
    before_digit = __shfl(before_digit, src, kWave);
    kk -= (int)before_digit;
    prefix |= (uint32_t)digit << shift;
    mask |= 255u << shift;
    lds_wait();
  }
  // every key above the k-th is taken, and the lowest-channel kk of those
  // equal to it; gathered in channel order
  const uint32_t kstar = prefix;
  const uint64_t below = (1ull << lane) - 1ull;
  int taken = 0, eq_seen = 0;
  for (int c0 = 0; c0 < C; c0 += kWave) {
    const int c = c0 + lane;
    const uint32_t key = c < C ? fkey(row[c]) : 0u;
    const bool eq = c < C && key == kstar;
    const uint64_t beq = __ballot(eq);
    const bool sel = (c < C && key > kstar) || (eq && eq_seen + __popcll(beq & below) < kk);
    const uint64_t bsel = __ballot(sel);
    if (sel && taken + __popcll(bsel & below) < P) {
      const int pos = taken + __popcll(bsel & below);
      lkey[pos] = key;
      lch[pos] = c;
    }
    taken += __popcll(bsel);
    eq_seen += __popcll(beq);
  }
  // bitonic sort of the k (padded to a power of two with entries that sort
  // last) into the canonical order
  for (int i = k + lane; i < P; i += kWave) {
    lkey[i] = 0u;
    lch[i] = INT_MAX;
  }
  lds_wait();
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = lane; i < P / 2; i += kWave) {
        const int lo = 2 * stride * (i / stride) + (i % stride), hi = lo + stride;
        const uint32_t ka = lkey[lo], kb = lkey[hi];
        const int ca = lch[lo], cb = lch[hi];
        // runs of `size` alternate between the canonical order and its reverse
        const bool forward = (lo & size) == 0;
        if (forward ? before(kb, cb, ka, ca) : before(ka, ca, kb, cb)) {
          lkey[lo] = kb;
          lch[lo] = cb;
          lkey[hi] = ka;
          lch[hi] = ca;
        }
      }
      lds_wait();
    }
  }
  for (int i = lane; i < k; i += kWave) {
    Sout[i] = lch[i];
    Wout[i] = fkey_value(lkey[i]);
  }
  lds_wait();
}

// EB experts of one image per workgroup of EB waves (a row each); DD >= the
// bottleneck width
template <int EB, int DD>
__global__ void __launch_bounds__(EB * kWave)
k_dyn_select(const float* __restrict__ h, const float* __restrict__ L, const float* __restrict__ q,
             const float* __restrict__ vT, int32_t* __restrict__ S, float* __restrict__ W, int C, int R, int k,
             int dd, int nblk) {
  extern __shared__ float sm[];
  float* rows = sm;              // [EB][C] the block's logit rows of this image
  float* qh = rows + EB * C;     // [EB][DD] q_e * h, zero past dd
  const int P = list_len(k);
  uint32_t* wsm = reinterpret_cast<uint32_t*>(qh + EB * DD) + (threadIdx.x >> 6) * (256 + 2 * P);
  uint32_t* hist = wsm;
  uint32_t* lkey = hist + 256;
  int32_t* lch = reinterpret_cast<int32_t*>(lkey + P);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t b = blockIdx.x / nblk;
  const int e0 = (int)(blockIdx.x % nblk) * EB;
  const int ne = min(EB, R - e0);
  for (int i = threadIdx.x; i < EB * DD; i += blockDim.x) {
    const int e = i / DD, t = i - e * DD;
    const float qv = q[(int64_t)min(e0 + e, R - 1) * dd + min(t, dd - 1)];
    const float hv = h[b * dd + min(t, dd - 1)];
    qh[i] = t < dd ? qv * hv : 0.f;
  }
  __syncthreads();
  // logits: a thread per channel, v_c in registers (from the transposed
  // embeddings vT[d][C], so a wave's reads of one t are consecutive), every
  // expert of the block
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    float vr[DD];
#pragma unroll
    for (int t = 0; t < DD; ++t) {
      const float x = vT[(int64_t)min(t, dd - 1) * C + c];
      vr[t] = t < dd ? x : 0.f;
    }
#pragma unroll 4
    for (int e = 0; e < EB; ++e) {
      float off = 0.f;
#pragma unroll
      for (int t = 0; t < DD; ++t) off += qh[e * DD + t] * vr[t];
      rows[e * C + c] = L[(int64_t)min(e0 + e, R - 1) * C + c] + off;
    }
  }
  __syncthreads();
  // each wave: one row
  for (int e = wv; e < ne; e += EB) {
    const int64_t item = b * R + e0 + e;
    select_row(rows + e * C, hist, lkey, lch, C, k, P, lane, S + item * k, W + item * k);
  }
}

// The same with the channel embeddings read once per workgroup: 16 waves hold
// v_c of CPT channels each in registers and walk nbp consecutive blocks of 16
// experts of one image, forming the block's rows in LDS (the same arithmetic,
// in the same order, as k_dyn_select) and selecting a row per wave.  Where
// 2 P <= 256 a wave's list overlaps its histogram (the histogram is dead once
// the k-th key is known).
constexpr int kSel2Waves = 16;
__host__ __device__ inline int wave_words2(int k) {
  return 2 * list_len(k) <= 256 ? 256 : 256 + 2 * list_len(k);
}

template <int DD, int CPT>
__global__ void __launch_bounds__(kSel2Waves * kWave)
k_dyn_select2(const float* __restrict__ h, const float* __restrict__ L, const float* __restrict__ q,
              const float* __restrict__ vT, int32_t* __restrict__ S, float* __restrict__ W, int C, int R, int k,
              int dd, int nblk, int nbp, int nsplit) {
  constexpr int EB = kSel2Waves;
  extern __shared__ float sm[];
  float* rows = sm;              // [EB][C]
  float* qh = rows + EB * C;     // [EB][DD]
  const int P = list_len(k);
  const int ww = wave_words2(k);
  uint32_t* hist = reinterpret_cast<uint32_t*>(qh + EB * DD) + (threadIdx.x >> 6) * ww;
  uint32_t* lkey = ww == 256 ? hist : hist + 256;
  int32_t* lch = reinterpret_cast<int32_t*>(lkey + P);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t b = blockIdx.x / nsplit;
  const int blk0 = (int)(blockIdx.x % nsplit) * nbp;
  const int blk1 = min(blk0 + nbp, nblk);
  float vr[CPT][DD];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int c = min((int)threadIdx.x + j * EB * kWave, C - 1);
#pragma unroll
    for (int t = 0; t < DD; ++t) {
      const float x = vT[(int64_t)min(t, dd - 1) * C + c];
      vr[j][t] = t < dd ? x : 0.f;
    }
  }
  for (int blk = blk0; blk < blk1; ++blk) {
    const int e0 = blk * EB;
    const int ne = min(EB, R - e0);
    for (int i = threadIdx.x; i < EB * DD; i += blockDim.x) {
      const int e = i / DD, t = i - e * DD;
      const float qv = q[(int64_t)min(e0 + e, R - 1) * dd + min(t, dd - 1)];
      const float hv = h[b * dd + min(t, dd - 1)];
      qh[i] = t < dd ? qv * hv : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int c = (int)threadIdx.x + j * EB * kWave;
      if (c < C) {
#pragma unroll 4
        for (int e = 0; e < EB; ++e) {
          float off = 0.f;
#pragma unroll
          for (int t = 0; t < DD; ++t) off += qh[e * DD + t] * vr[j][t];
          rows[e * C + c] = L[(int64_t)min(e0 + e, R - 1) * C + c] + off;
        }
      }
    }
    __syncthreads();
    if (wv < ne) {
      const int64_t item = b * R + e0 + wv;
      select_row(rows + wv * C, hist, lkey, lch, C, k, P, lane, S + item * k, W + item * k);
    }
    __syncthreads();  // rows and qh free for the next block
  }
}

// ---------------------------------------------------------------- U(X)
// A workgroup per image: the channels in none of the image's supports, in
// ascending order, by a block-wide compaction.
__global__ void __launch_bounds__(1024)
k_dyn_uncovered(const int32_t* __restrict__ S, int32_t* __restrict__ U, int32_t* __restrict__ nU, int C, int R,
                int k) {
  extern __shared__ unsigned char cov[];  // [C] flags, then 16 wave counts
  int32_t* wcnt = reinterpret_cast<int32_t*>(cov + ((C + 15) & ~15));
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int c = threadIdx.x; c < C; c += blockDim.x) cov[c] = 0;
  __syncthreads();
  const int64_t n = (int64_t)R * k;
#pragma unroll 8
  for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
    const int32_t c = S[b * n + j];
    if ((uint32_t)c < (uint32_t)C) cov[c] = 1;
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
  int base = 0;
  for (int c0 = 0; c0 < C; c0 += blockDim.x) {
    const int c = c0 + threadIdx.x;
    const bool f = c < C && !cov[c];
    const uint64_t bf = __ballot(f);
    if (lane == 0) wcnt[wv] = __popcll(bf);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wv; ++w) off += wcnt[w];
    if (f) U[b * C + off + __popcll(bf & below)] = c;
    int tot = 0;
    for (int w = 0; w < nw; ++w) tot += wcnt[w];
    base += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) nU[b] = base;
}

// ---------------------------------------------------------------- gate
// A wave per (image, routed expert): z at the example's support, the gate's
// temperature, and the coefficients from the example's logits there (the
// library's coefficient operations; the largest scaled logit from the
// largest logit, as 1/tau > 0).
__global__ void __launch_bounds__(kDynThreads)
k_dyn_gate(const float* __restrict__ d, const int32_t* __restrict__ S, const float* __restrict__ W,
           moce_gate_params g, float* __restrict__ tau, float* __restrict__ alpha, int64_t B, int C, int R, int k) {
  __shared__ float zsm[kDynWaves][kDynMaxK];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t item = (int64_t)blockIdx.x * kDynWaves + wv;
  if (item >= B * R) return;  // whole waves; no block barrier below
  const int64_t b = item / R;
  const int e = (int)(item - b * R);
  const int32_t* s = S + item * k;
  const float* w = W + item * k;
  float* z = zsm[wv];
  for (int i = lane; i < k; i += kWave) z[i] = d[b * C + min(max(s[i], 0), C - 1)];
  lds_wait();
  float t;
  if (g.kind == MOCE_GATE_SOFTPLUS_LINEAR) {
    float acc = 0.f;
    for (int i = lane; i < k; i += kWave) acc += g.a[(int64_t)e * k + i] * z[i];
    t = softplusf(wave_sum(acc) + g.c[e]) + 1e-3f;
  } else {
    float acc = 0.f;
    for (int j = lane; j < k; j += kWave) {
      float hj = g.b1[j];
      for (int i = 0; i < k; ++i) hj += g.W1[(int64_t)j * k + i] * z[i];
      acc += g.w2[j] * fmaxf(hj, 0.f);
    }
    const float gg = wave_sum(acc) + g.b2;
    t = g.tau_min + (g.tau_max - g.tau_min) / (1.f + expf(-gg));
  }
  const float rt = 1.f / t;
  float wm = -INFINITY;
  for (int i = lane; i < k; i += kWave) wm = fmaxf(wm, w[i]);
  const float m = coef_z(wave_max(wm), rt);
  float zs = 0.f;
  for (int i = lane; i < k; i += kWave) zs += coef_e(coef_z(w[i], rt), m);
  const float rzs = 1.f / wave_sum(zs);
  for (int i = lane; i < k; i += kWave) alpha[item * k + i] = coef_alpha(coef_e(coef_z(w[i], rt), m), rzs);
  if (lane == 0) tau[item] = t;
}

// ---------------------------------------------------------------- mix
template <typename T> __device__ __forceinline__ float ld(const T* p);
template <> __device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <typename T> __device__ __forceinline__ void st(T* p, float v);
template <> __device__ __forceinline__ void st<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16(v); }

// A workgroup per (image, TP positions): the tile of every channel staged in
// LDS as float [C][TP]; a thread per output channel accumulates its TP
// positions over the example's support (or over U(X) for the residual).
constexpr int kDynTP = 8;

template <typename T, bool NHWC>
__global__ void __launch_bounds__(kDynThreads)
k_dyn_mix(const T* __restrict__ x, const int32_t* __restrict__ S, const float* __restrict__ alpha,
          const int32_t* __restrict__ U, const int32_t* __restrict__ nU, T* __restrict__ y, int C, int HW, int E,
          int k, int ntiles) {
  extern __shared__ float xs[];  // [C][kDynTP]
  const int R = E - 1;
  const int64_t b = blockIdx.x / ntiles;
  const int p0 = (int)(blockIdx.x % ntiles) * kDynTP;
  const T* xb = x + b * (int64_t)C * HW;
  for (int idx = threadIdx.x; idx < C * kDynTP; idx += blockDim.x) {
    int c, j;
    if (NHWC) {  // consecutive threads on consecutive channels of one position
      j = idx / C;
      c = idx - j * C;
    } else {     // consecutive threads on consecutive positions of one channel
      c = idx / kDynTP;
      j = idx - c * kDynTP;
    }
    const int p = min(p0 + j, HW - 1);
    xs[c * kDynTP + j] = ld<T>(NHWC ? xb + (int64_t)p * C + c : xb + (int64_t)c * HW + p);
  }
  __syncthreads();
  for (int o = threadIdx.x; o < E; o += blockDim.x) {
    float acc[kDynTP];
#pragma unroll
    for (int j = 0; j < kDynTP; ++j) acc[j] = 0.f;
    if (o < R) {
      const int64_t item = b * R + o;
#pragma unroll 8
      for (int i = 0; i < k; ++i) {
        const float a = alpha[item * k + i];
        const float4* r = reinterpret_cast<const float4*>(xs + min(max(S[item * k + i], 0), C - 1) * kDynTP);
#pragma unroll
        for (int j4 = 0; j4 < kDynTP / 4; ++j4) {
          const float4 v = r[j4];
          acc[4 * j4] += a * v.x;
          acc[4 * j4 + 1] += a * v.y;
          acc[4 * j4 + 2] += a * v.z;
          acc[4 * j4 + 3] += a * v.w;
        }
      }
    } else {
      const int n = nU[b];
#pragma unroll 8
      for (int u = 0; u < n; ++u) {
        const float4* r = reinterpret_cast<const float4*>(xs + U[b * C + u] * kDynTP);
#pragma unroll
        for (int j4 = 0; j4 < kDynTP / 4; ++j4) {
          const float4 v = r[j4];
          acc[4 * j4] += v.x;
          acc[4 * j4 + 1] += v.y;
          acc[4 * j4 + 2] += v.z;
          acc[4 * j4 + 3] += v.w;
        }
      }
      const float inv = n > 0 ? 1.f / (float)n : 0.f;
#pragma unroll
      for (int j = 0; j < kDynTP; ++j) acc[j] *= inv;
    }
#pragma unroll
    for (int j = 0; j < kDynTP; ++j) {
      const int p = p0 + j;
      if (p < HW) st<T>(NHWC ? y + (b * HW + p) * (int64_t)E + o : y + (b * E + o) * (int64_t)HW + p, acc[j]);
    }
  }
}

// experts (and waves) per selection workgroup: 8 where two workgroups fit
// a CU's LDS, else as many as one fits
size_t select_lds(const Shape& sh, int eb, int DD) {
  return ((size_t)eb * sh.C + (size_t)eb * DD) * 4 + (size_t)eb * wave_words(sh.k) * 4;
}
int select_eb(const Shape& sh, int DD) {
  for (int eb : {8, 4, 2, 1})
    if (2 * select_lds(sh, eb, DD) <= kDynLds) return eb;
  for (int eb : {8, 4, 2, 1})
    if (select_lds(sh, eb, DD) <= kDynLds) return eb;
  return 0;
}

size_t select2_lds(const Shape& sh, int DD) {
  return ((size_t)kSel2Waves * sh.C + (size_t)kSel2Waves * DD + (size_t)kSel2Waves * wave_words2(sh.k)) * 4;
}
// channels per thread of k_dyn_select2, or 0 where its registers or LDS do
// not hold the shape
int select2_cpt(const Shape& sh, int DD) {
  const int cpt = (int)((sh.C + kSel2Waves * kWave - 1) / (kSel2Waves * kWave));
  if (cpt * DD > 64 || select2_lds(sh, DD) > kDynLds) return 0;
  return cpt;
}

template <int DD>
hipError_t launch_select_dd(const Shape& sh, const float* h, const float* L, const float* q, const float* vT,
                            int32_t* S, float* W, int dd, hipStream_t st) {
  using K = void (*)(const float*, const float*, const float*, const float*, int32_t*, float*, int, int, int, int,
                     int);
  using K2 = void (*)(const float*, const float*, const float*, const float*, int32_t*, float*, int, int, int, int,
                      int, int, int);
  // the register-held embeddings where the per-block kernel's LDS limits its
  // blocks below eight experts (each block then reads every embedding for
  // fewer than eight rows)
  const int cpt = select_eb(sh, DD) < 8 ? select2_cpt(sh, DD) : 0;
  if (cpt > 0) {
    // blocks of 16 experts, nbp per workgroup, for about two workgroups per CU
    const int nblk = (sh.R + kSel2Waves - 1) / kSel2Waves;
    int cus = 256, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    const int64_t total = sh.B * nblk;
    const int nbp = (int)std::max<int64_t>(1, std::min<int64_t>(nblk, total / (2 * cus)));
    const int nsplit = (nblk + nbp - 1) / nbp;
    const size_t lds = select2_lds(sh, DD);
    const K2 kern = cpt == 1 ? k_dyn_select2<DD, 1> : k_dyn_select2<DD, (DD <= 32 ? 2 : 1)>;
    if (cpt == 2 && DD > 32) return hipErrorInvalidValue;
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)(sh.B * nsplit)), dim3(kSel2Waves * kWave), lds, st, h, L, q, vT, S, W,
                       (int)sh.C, sh.R, sh.k, dd, nblk, nbp, nsplit);
    return hipGetLastError();
  }
  const int eb = select_eb(sh, DD);
  if (eb == 0) return hipErrorInvalidValue;
  const int nblk = (sh.R + eb - 1) / eb;
  const size_t lds = select_lds(sh, eb, DD);
  const K kern = eb == 8 ? k_dyn_select<8, DD> : eb == 4 ? k_dyn_select<4, DD> : eb == 2 ? k_dyn_select<2, DD>
                                                                                       : k_dyn_select<1, DD>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)(sh.B * nblk)), dim3(eb * kWave), lds, st, h, L, q, vT, S, W, (int)sh.C,
                     sh.R, sh.k, dd, nblk);
  return hipGetLastError();
}

}  // namespace

bool dynamic_supported(const Shape& sh, int dd) {
  if (dd < 1 || dd > kDynMaxD || sh.k > kDynMaxK) return false;
  if (sh.C > kDynMaxC) return false;
  return select_eb(sh, dd <= 32 ? 32 : 64) > 0;
}

hipError_t launch_dynamic(const Shape& sh, const void* x, const float* L, const moce_router& r,
                          const moce_gate_params& g, void* y, float* d, float* h, float* vT, int32_t* S, float* W,
                          int32_t* U, int32_t* nU, float* tau, float* alpha, hipStream_t st) {
  hipError_t e = launch_pool(sh, x, d, st);
  if (e != hipSuccess) return e;
  if (sh.R > 0) {
    const int64_t waves = sh.B * r.d;
    hipLaunchKernelGGL(k_dyn_router, dim3((unsigned)((waves + kDynWaves - 1) / kDynWaves)), dim3(kDynThreads), 0,
                       st, d, r.Wh, r.bh, h, sh.B, (int)sh.C, r.d);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_dyn_transpose, dim3((unsigned)((sh.C + 31) / 32), (unsigned)((r.d + 31) / 32)), dim3(1024),
                       0, st, r.v, vT, (int)sh.C, r.d);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = r.d <= 32 ? launch_select_dd<32>(sh, h, L, r.q, vT, S, W, r.d, st)
                  : launch_select_dd<64>(sh, h, L, r.q, vT, S, W, r.d, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_dyn_uncovered, dim3((unsigned)sh.B), dim3(1024), ((sh.C + 15) & ~15) + 16 * 4, st, S, U, nU,
                     (int)sh.C, sh.R, sh.k);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (sh.R > 0) {
    const int64_t items = sh.B * sh.R;
    hipLaunchKernelGGL(k_dyn_gate, dim3((unsigned)((items + kDynWaves - 1) / kDynWaves)), dim3(kDynThreads), 0, st, d,
                       S, W, g, tau, alpha, sh.B, (int)sh.C, sh.R, sh.k);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (tilemix_dynamic_eligible(sh)) return launch_tilemix_dynamic(sh, x, S, alpha, U, nU, y, st);
  const int ntiles = (int)((sh.HW + kDynTP - 1) / kDynTP);
  const size_t lds = (size_t)sh.C * kDynTP * sizeof(float);
  const unsigned grid = (unsigned)(sh.B * ntiles);
  using KB = void (*)(const uint16_t*, const int32_t*, const float*, const int32_t*, const int32_t*, uint16_t*, int,
                      int, int, int, int);
  using KF = void (*)(const float*, const int32_t*, const float*, const int32_t*, const int32_t*, float*, int, int,
                      int, int, int);
  if (sh.elem == MOCE_BF16) {
    const KB kern = sh.layout == MOCE_NHWC ? k_dyn_mix<uint16_t, true> : k_dyn_mix<uint16_t, false>;
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kDynThreads), lds, st, static_cast<const uint16_t*>(x), S, alpha, U, nU,
                       static_cast<uint16_t*>(y), (int)sh.C, (int)sh.HW, sh.E, sh.k, ntiles);
  } else {
    const KF kern = sh.layout == MOCE_NHWC ? k_dyn_mix<float, true> : k_dyn_mix<float, false>;
    e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kDynThreads), lds, st, static_cast<const float*>(x), S, alpha, U, nU,
                       static_cast<float*>(y), (int)sh.C, (int)sh.HW, sh.E, sh.k, ntiles);
  }
  return hipGetLastError();
}

}  // namespace moce

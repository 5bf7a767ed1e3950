// Gradients of the static layer (Secs. 3.2-3.4) and of the coverage loss
// (Sec. 3.4 Eq. 7).
//
// With dy the gradient of the loss with respect to y, the layer's backward is
//   dalpha[b][e][i] = sum_p dy[b][e][p] x[b][s_ei][p]                (Eq. 5)
//   dz_i  = alpha_i (dalpha_i - sum_j alpha_j dalpha_j)               (Eq. 4)
//   dw[e][i]  = sum_b dz_bei / tau_be
//   dtau_be   = -sum_i dz_bei w_ei / tau_be^2
//   the gate's parameters from dtau; its inputs z_i = d[b][s_ei] from dtau
//   dx[b][c][p] = sum_{(e,i): s_ei = c} alpha_bei dy[b][e][p]
//               + [c uncovered] dy[b][E-1][p] / |U|                    (Eq. 6)
//               + dd[b][c] / HW                                        (GAP)
// where dd[b][c] sums the gate-input gradients of every support entry on c.
//
// Launches:
//  - pooling and the forward's gate (pool.hip, gate.hip): d, the softmax
//    statistics and the coefficients;
//  - the inverse support map (channel -> support entries), rebuilt per call
//    from the prepared rows: counts, one scan (which also counts |U|), a fill
//    and a per-channel sort, so the sums over a channel's entries run in a
//    fixed order;
//  - dalpha (the sampled product of dy and x; the matrix-core kernel of
//    bwdmfma.hip where it applies, a wave per (image, expert) elsewhere);
//  - a wave per (image, expert) for the row sums, dtau and the
//    softplus-linear gate's dg; the MLP gate's rows in blocks (below);
//  - a thread per (expert, position) summing dw and the gate's slopes over
//    the images;
//  - dd (a thread per (image, channel)) and dx (the matrix-core kernel of
//    bwdmfma.hip where it applies, a thread per element elsewhere).
#include <algorithm>
#include <climits>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kBwThreads = 256;
constexpr int kBwWaves = kBwThreads / kWave;
constexpr int kBwMaxK = 1024;     // a support row in registers, 16 entries per lane
constexpr int kCovMaxC = 32768;   // a logit row's support positions in LDS

template <typename T> __device__ __forceinline__ float ld(const T* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<uint16_t>(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
template <typename T> __device__ __forceinline__ void st_elem(T* p, int64_t i, float v);
template <> __device__ __forceinline__ void st_elem<float>(float* p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_elem<uint16_t>(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }

// element (b, channel c of nc, position p) of an NCHW or channels-last tensor
template <bool NHWC>
__device__ __forceinline__ int64_t at(int64_t b, int64_t c, int64_t p, int64_t nc, int64_t HW) {
  return NHWC ? (b * HW + p) * nc + c : (b * nc + c) * HW + p;
}

__device__ __forceinline__ float alpha_of(float w, float rt, float m, float rzs) {
  return coef_alpha(coef_e(coef_z(w, rt), m), rzs);
}

// ---------------------------------------------------------------- inverse support map
__global__ void k_bw_fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_inv_count(const int32_t* __restrict__ s, int64_t n, int32_t* __restrict__ cnt) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) atomicAdd(&cnt[s[t]], 1);
}

// One workgroup: off[c] = sum_{c' < c} cnt[c'], off[C] = total; cur = off;
// nU = the number of channels with no entry.
__global__ void __launch_bounds__(1024)
k_inv_scan(const int32_t* __restrict__ cnt, int32_t* __restrict__ off, int32_t* __restrict__ cur,
           int32_t* __restrict__ nU, int C) {
  __shared__ int32_t part[1024];
  __shared__ int32_t zpart[1024];
  const int t = threadIdx.x;
  const int per = (C + 1023) / 1024;
  const int c0 = min(t * per, C), c1 = min(c0 + per, C);
  int32_t sum = 0, zeros = 0;
  for (int c = c0; c < c1; ++c) {
    sum += cnt[c];
    zeros += cnt[c] == 0;
  }
  part[t] = sum;
  zpart[t] = zeros;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {  // inclusive scan of the partial sums
    const int32_t v = t >= o ? part[t - o] : 0;
    const int32_t z = t >= o ? zpart[t - o] : 0;
    __syncthreads();
    part[t] += v;
    zpart[t] += z;
    __syncthreads();
  }
  int32_t run = t > 0 ? part[t - 1] : 0;
  for (int c = c0; c < c1; ++c) {
    off[c] = run;
    cur[c] = run;
    run += cnt[c];
  }
  if (t == 1023) {
    off[C] = part[1023];
    *nU = zpart[1023];
  }
}

__global__ void k_inv_fill(const int32_t* __restrict__ s, int64_t n, int32_t* __restrict__ cur,
                           int32_t* __restrict__ inv) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) inv[atomicAdd(&cur[s[t]], 1)] = (int32_t)t;
}

// each channel's entries ascending (by expert, as a row holds a channel once):
// a wave per channel; up to 64 entries by rank (each entry's place is the
// number of smaller ones), longer lists by insertion on one lane
__global__ void __launch_bounds__(256)
k_inv_sort(const int32_t* __restrict__ off, int32_t* __restrict__ inv, int C) {
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (c >= C) return;
  const int lane = threadIdx.x & 63;
  const int a = off[c], n = off[c + 1] - a;
  if (n <= 64) {
    const int32_t v = lane < n ? inv[a + lane] : INT_MAX;
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += __shfl(v, j) < v;
    if (lane < n) inv[a + rank] = v;
    return;
  }
  if (lane != 0) return;
  for (int j = a + 1; j < a + n; ++j) {
    const int32_t v = inv[j];
    int q = j - 1;
    while (q >= a && inv[q] > v) {
      inv[q + 1] = inv[q];
      --q;
    }
    inv[q + 1] = v;
  }
}

// ---------------------------------------------------------------- dalpha, generic
// A wave per (image, routed expert); lanes over support positions.
template <typename T, bool NHWC>
__global__ void __launch_bounds__(kBwThreads)
k_bw_dalpha(const T* __restrict__ x, const T* __restrict__ dy, const int32_t* __restrict__ s,
            float* __restrict__ dal, int64_t B, int C, int E, int R, int k, int HW) {
  const int64_t row = (int64_t)blockIdx.x * kBwWaves + (threadIdx.x >> 6);
  if (row >= B * R) return;
  const int lane = threadIdx.x & 63;
  const int64_t b = row / R;
  const int e = (int)(row - b * R);
  for (int i0 = 0; i0 < k; i0 += kWave) {
    const int i = i0 + lane;
    const int c = i < k ? s[(int64_t)e * k + i] : 0;
    float acc = 0.f;
    for (int p = 0; p < HW; ++p) {
      const float g = ld<T>(dy, at<NHWC>(b, e, p, E, HW));
      acc += g * ld<T>(x, at<NHWC>(b, c, p, C, HW));
    }
    if (i < k) dal[row * k + i] = acc;
  }
}

// ---------------------------------------------------------------- rows: S1, dtau, dg
// A wave per (image, routed expert); dalpha arrives as nsplit partial sums,
// whose total replaces the first.  S1 = sum_i alpha_i dalpha_i; with
// Aw = sum_i alpha_i w_i, sum_i dz_i w_i = sum_i alpha_i (dalpha_i - S1) (w_i - Aw),
// centred twice so that nothing cancels; dtau = -that / tau^2 (rt = 1/tau).
// Softplus-linear gate: g = c_e + sum_i a_ei z_i, dg = dtau sigmoid(g).
template <int NPL>
__global__ void __launch_bounds__(kBwThreads)
k_bw_rows(float* __restrict__ dal, const float* __restrict__ w, const float* __restrict__ stats,
          const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ a,
          const float* __restrict__ cc, float* __restrict__ S1o, float* __restrict__ dtau_o,
          float* __restrict__ dg_o, int64_t B, int C, int R, int k, int nsplit) {
  const int64_t row = (int64_t)blockIdx.x * kBwWaves + (threadIdx.x >> 6);
  if (row >= B * R) return;
  const int lane = threadIdx.x & 63;
  const int64_t b = row / R;
  const int e = (int)(row - b * R);
  const int64_t n = B * R;
  const float rt = stats[row], m = stats[n + row], rzs = stats[2 * n + row];
  float al[NPL], da[NPL], wv[NPL];
  float s1 = 0.f, aw = 0.f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int i = lane + j * kWave;
    al[j] = 0.f;
    da[j] = 0.f;
    wv[j] = 0.f;
    if (i < k) {
      wv[j] = w[(int64_t)e * k + i];
      al[j] = alpha_of(wv[j], rt, m, rzs);
      da[j] = dal[row * k + i];
      if (nsplit > 1) {  // partial sums along the positions: total into the first block
        for (int sp = 1; sp < nsplit; ++sp) da[j] += dal[(sp * n + row) * k + i];
        dal[row * k + i] = da[j];
      }
      s1 += al[j] * da[j];
      aw += al[j] * wv[j];
    }
  }
  s1 = wave_sum(s1);
  aw = wave_sum(aw);
  float t = 0.f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) t += al[j] * (da[j] - s1) * (wv[j] - aw);
  t = wave_sum(t);
  const float dtau = -t * rt * rt;
  float dg = 0.f;
  if (a) {
    float g = 0.f;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int i = lane + j * kWave;
      if (i < k) g += a[(int64_t)e * k + i] * d[b * C + s[(int64_t)e * k + i]];
    }
    g = wave_sum(g) + cc[e];
    dg = dtau / (1.f + expf(-g));
  }
  if (lane == 0) {
    S1o[row] = s1;
    dtau_o[row] = dtau;
    if (a) dg_o[row] = dg;
  }
}

// ---------------------------------------------------------------- sums over images
// Partial sums over groups of images (grid.y = group g of gs images), a thread
// per (routed expert, support position):
//   dw[e][i] = sum_b alpha_bei (dalpha_bei - S1_be) rt_be,
//   da[e][i] = sum_b dg_be d[b][s_ei]  (softplus-linear gate only),
// and, on the threads of position 0, dc[e] = sum_b dg_be; then one pass sums
// the groups in order.
__global__ void __launch_bounds__(kBwThreads)
k_bw_sums(const float* __restrict__ dal, const float* __restrict__ w, const float* __restrict__ stats,
          const float* __restrict__ S1, const float* __restrict__ dg, const float* __restrict__ d,
          const int32_t* __restrict__ s, float* __restrict__ pdw, float* __restrict__ pda, float* __restrict__ pdc,
          int64_t B, int C, int R, int k, int gs, bool gate_sums) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t rk = (int64_t)R * k;
  if (t >= rk) return;
  const int g = blockIdx.y;
  const int e = (int)(t / k);
  const int64_t n = B * R;
  const float wv = w[t];
  const int c = s[t];
  float sw = 0.f, sa = 0.f, sc = 0.f;
  const int64_t b1 = min<int64_t>(B, (int64_t)(g + 1) * gs);
  for (int64_t b = (int64_t)g * gs; b < b1; ++b) {
    const int64_t row = b * R + e;
    const float rt = stats[row];
    const float al = alpha_of(wv, rt, stats[n + row], stats[2 * n + row]);
    sw += al * (dal[b * rk + t] - S1[row]) * rt;
    if (gate_sums) {
      sa += dg[row] * d[b * C + c];
      sc += dg[row];
    }
  }
  pdw[g * rk + t] = sw;
  if (gate_sums) {
    pda[g * rk + t] = sa;
    if (t % k == 0) pdc[(int64_t)g * R + e] = sc;
  }
}

__global__ void k_bw_sums_reduce(const float* __restrict__ pdw, const float* __restrict__ pda,
                                 const float* __restrict__ pdc, int ng, int64_t rk, int R, float* __restrict__ dw,
                                 float* __restrict__ da, float* __restrict__ dc) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < rk) {
    float sw = 0.f, sa = 0.f;
#pragma unroll 8
    for (int g = 0; g < ng; ++g) {
      sw += pdw[g * rk + t];
      if (da) sa += pda[g * rk + t];
    }
    dw[t] = sw;
    if (da) da[t] = sa;
  }
  if (dc && t < R) {
    float sc = 0.f;
#pragma unroll 8
    for (int g = 0; g < ng; ++g) sc += pdc[(int64_t)g * R + t];
    dc[t] = sc;
  }
}

// ---------------------------------------------------------------- dd
// dd[b][c] = sum over the entries (e, i) on channel c of the gate-input
// gradient: dg_be a_ei (softplus-linear) or dzg[b][e][i] (MLP).
__global__ void __launch_bounds__(kBwThreads)
k_bw_dd(const int32_t* __restrict__ off, const int32_t* __restrict__ inv, const float* __restrict__ dg,
        const float* __restrict__ a, const float* __restrict__ dzg, float* __restrict__ dd, int64_t B, int C, int R,
        int k) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= B * C) return;
  const int64_t b = t / C;
  const int c = (int)(t - b * C);
  const int64_t rk = (int64_t)R * k;
  float acc = 0.f;
#pragma unroll 8
  for (int j = off[c]; j < off[c + 1]; ++j) {
    const int ent = inv[j];
    if (a)
      acc += dg[b * R + ent / k] * a[ent];
    else
      acc += dzg[b * rk + ent];
  }
  dd[t] = acc;
}

// ---------------------------------------------------------------- dx, generic
// A thread per element of dx: the channel's entries in inverse-map order,
// then the residual share and the descriptor term.
template <typename T, bool NHWC>
__global__ void __launch_bounds__(kBwThreads)
k_bw_dx(const T* __restrict__ dy, const float* __restrict__ alpha, const int32_t* __restrict__ off,
        const int32_t* __restrict__ inv, const int32_t* __restrict__ nUp, const float* __restrict__ dd,
        T* __restrict__ dx, int64_t B, int C, int E, int R, int k, int HW) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = B * C * (int64_t)HW;
  if (t >= total) return;
  int64_t b, c, p;
  if (NHWC) {
    c = t % C;
    const int64_t r = t / C;
    p = r % HW;
    b = r / HW;
  } else {
    p = t % HW;
    const int64_t r = t / HW;
    c = r % C;
    b = r / C;
  }
  const int64_t rk = (int64_t)R * k;
  float acc = 0.f;
  const int j0 = off[c], j1 = off[c + 1];
  for (int j = j0; j < j1; ++j) {
    const int ent = inv[j];
    const int e = ent / k;
    acc += alpha[b * rk + ent] * ld<T>(dy, at<NHWC>(b, e, p, E, HW));
  }
  if (j0 == j1) acc += ld<T>(dy, at<NHWC>(b, R, p, E, HW)) / (float)*nUp;
  if (R > 0) acc += dd[b * C + c] / (float)HW;
  st_elem<T>(dx, t, acc);
}

// ---------------------------------------------------------------- the MLP gate
// Rows r = (b, e) in blocks of kMlpBwRows per workgroup, W1 in LDS.  Per row:
// z_i = d[b][s_ei], hpre = W1 z + b1, h = ReLU(hpre), g = w2 . h + b2,
// sigma = sigmoid(g), dg = dtau (tmax - tmin) sigma (1 - sigma),
// dh_j = dg w2_j [hpre_j > 0], dzg_i = sum_j W1[j][i] dh_j (written per row);
// the workgroup accumulates dW1 += dh z^T, db1 += dh, dw2 += dg h, db2 += dg
// and writes them as one partial per workgroup.
constexpr int kMlpBwRows = 16;
constexpr int kMlpBwMaxK = 128;

__global__ void __launch_bounds__(kBwThreads)
k_bw_mlp(const float* __restrict__ d, const int32_t* __restrict__ s, const float* __restrict__ dtau,
         const float* __restrict__ W1, const float* __restrict__ b1, const float* __restrict__ w2, float b2,
         float tmin, float tmax, float* __restrict__ dzg, float* __restrict__ part, int64_t B, int C, int R, int k) {
  extern __shared__ float lds[];
  float* w1s = lds;                                 // [k][k]
  float* zs = w1s + k * k;                          // [rows][k]
  float* hs = zs + kMlpBwRows * k;                  // [rows][k]: hpre, then dh
  float* gs = hs + kMlpBwRows * k;                  // [rows]: dg
  const int tid = threadIdx.x;
  for (int q = tid; q < k * k; q += kBwThreads) w1s[q] = W1[q];
  const int kk = k * k;
  // partial dW1 in registers: thread owns entries q = tid + j * 256
  constexpr int kPer = kMlpBwMaxK * kMlpBwMaxK / kBwThreads;
  float pw[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) pw[j] = 0.f;
  float pb1 = 0.f, pw2 = 0.f, pb2 = 0.f;  // thread tid < k owns unit tid; thread 0 owns b2
  const int64_t nrows = B * R;
  const int64_t nblk = (nrows + kMlpBwRows - 1) / kMlpBwRows;
  const float span = tmax - tmin;
  for (int64_t blk = blockIdx.x; blk < nblk; blk += gridDim.x) {
    const int64_t r0 = blk * kMlpBwRows;
    const int nr = (int)min((int64_t)kMlpBwRows, nrows - r0);
    __syncthreads();
    for (int q = tid; q < kMlpBwRows * k; q += kBwThreads) {
      const int rr = q / k, i = q - rr * k;
      float z = 0.f;
      if (rr < nr) {
        const int64_t row = r0 + rr;
        const int64_t b = row / R;
        const int e = (int)(row - b * R);
        z = d[b * C + s[(int64_t)e * k + i]];
      }
      zs[q] = z;
    }
    __syncthreads();
    for (int q = tid; q < kMlpBwRows * k; q += kBwThreads) {  // hpre
      const int rr = q / k, j = q - rr * k;
      float acc = b1[j];
      for (int i = 0; i < k; ++i) acc += w1s[j * k + i] * zs[rr * k + i];
      hs[q] = acc;
    }
    __syncthreads();
    {  // g, sigma, dg: a wave per row
      const int wv = tid >> 6, lane = tid & 63;
      for (int rr = wv; rr < kMlpBwRows; rr += kBwWaves) {
        float g = 0.f;
        for (int j = lane; j < k; j += kWave) g += w2[j] * fmaxf(hs[rr * k + j], 0.f);
        g = wave_sum(g) + b2;
        const float sg = 1.f / (1.f + expf(-g));
        const float dg = rr < nr ? dtau[r0 + rr] * span * sg * (1.f - sg) : 0.f;
        if (lane == 0) gs[rr] = dg;
      }
    }
    __syncthreads();
    if (tid < k) {  // dw2, db1 partials; then hs becomes dh
      const int j = tid;
      for (int rr = 0; rr < nr; ++rr) {
        const float hp = hs[rr * k + j];
        const float dg = gs[rr];
        pw2 += dg * fmaxf(hp, 0.f);
        const float dh = hp > 0.f ? dg * w2[j] : 0.f;
        pb1 += dh;
        hs[rr * k + j] = dh;
      }
      for (int rr = nr; rr < kMlpBwRows; ++rr) hs[rr * k + j] = 0.f;
    }
    if (tid == 0)
      for (int rr = 0; rr < nr; ++rr) pb2 += gs[rr];
    __syncthreads();
    for (int q = tid; q < kMlpBwRows * k; q += kBwThreads) {  // dzg = W1^T dh
      const int rr = q / k, i = q - rr * k;
      if (rr >= nr) continue;
      float acc = 0.f;
      for (int j = 0; j < k; ++j) acc += w1s[j * k + i] * hs[rr * k + j];
      dzg[(r0 + rr) * k + i] = acc;
    }
#pragma unroll
    for (int jj = 0; jj < kPer; ++jj) {  // dW1 += dh z^T
      const int q = tid + jj * kBwThreads;
      if (q < kk) {
        const int j = q / k, i = q - j * k;
        float acc = pw[jj];
        for (int rr = 0; rr < nr; ++rr) acc += hs[rr * k + j] * zs[rr * k + i];
        pw[jj] = acc;
      }
    }
  }
  // partial layout per workgroup: [k*k dW1][k db1][k dw2][1 db2]
  float* out = part + (int64_t)blockIdx.x * (kk + 2 * k + 1);
#pragma unroll
  for (int jj = 0; jj < kPer; ++jj) {
    const int q = tid + jj * kBwThreads;
    if (q < kk) out[q] = pw[jj];
  }
  if (tid < k) {
    out[kk + tid] = pb1;
    out[kk + k + tid] = pw2;
  }
  if (tid == 0) out[kk + 2 * k] = pb2;
}

// sums the per-workgroup partials into dW1, db1, dw2, db2
__global__ void k_bw_mlp_reduce(const float* __restrict__ part, int nparts, int k, float* __restrict__ dW1,
                                float* __restrict__ db1, float* __restrict__ dw2, float* __restrict__ db2) {
  const int n = k * k + 2 * k + 1;
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= n) return;
  float acc = 0.f;
  for (int j = 0; j < nparts; ++j) acc += part[(int64_t)j * n + q];
  if (q < k * k)
    dW1[q] = acc;
  else if (q < k * k + k)
    db1[q - k * k] = acc;
  else if (q < k * k + 2 * k)
    dw2[q - k * k - k] = acc;
  else
    *db2 = acc;
}

// ---------------------------------------------------------------- coverage loss
// Row statistics of the full logits: m_e = max_c L[e][c], Z_e = sum_c exp(L - m_e).
__global__ void __launch_bounds__(kBwThreads)
k_cov_rows(const float* __restrict__ L, float* __restrict__ mz, int C) {
  __shared__ float red[kBwWaves];
  const int e = blockIdx.x;
  const float* row = L + (int64_t)e * C;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  float m = -INFINITY;
  for (int c = tid; c < C; c += kBwThreads) m = fmaxf(m, row[c]);
  m = wave_max(m);
  if (lane == 0) red[wv] = m;
  __syncthreads();
  m = red[0];
  for (int j = 1; j < kBwWaves; ++j) m = fmaxf(m, red[j]);
  __syncthreads();
  float z = 0.f;
  for (int c = tid; c < C; c += kBwThreads) z += expf(row[c] - m);
  z = wave_sum(z);
  if (lane == 0) red[wv] = z;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
    for (int j = 0; j < kBwWaves; ++j) t += red[j];
    mz[2 * e] = m;
    mz[2 * e + 1] = t;
  }
}

// u[c] = (1/R) sum_e exp(L[e][c] - m_e) / Z_e
__global__ void k_cov_cols(const float* __restrict__ L, const float* __restrict__ mz, float* __restrict__ u, int R,
                           int C) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  float acc = 0.f;
  for (int e = 0; e < R; ++e) acc += expf(L[(int64_t)e * C + c] - mz[2 * e]) / mz[2 * e + 1];
  u[c] = acc / (float)R;
}

// One workgroup: ub = mean u, num = sum (u - ub)^2, den = ub^2 + eps;
// sc = {ub, num, den}; loss = num / den.
__global__ void __launch_bounds__(1024)
k_cov_scalar(const float* __restrict__ u, int C, float eps, float* __restrict__ sc, float* __restrict__ loss) {
  __shared__ float red[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  float s = 0.f;
  for (int c = tid; c < C; c += 1024) s += u[c];
  s = wave_sum(s);
  if (lane == 0) red[wv] = s;
  __syncthreads();
  float tot = 0.f;
  for (int j = 0; j < 16; ++j) tot += red[j];
  const float ub = tot / (float)C;
  __syncthreads();
  float q = 0.f;
  for (int c = tid; c < C; c += 1024) {
    const float dv = u[c] - ub;
    q += dv * dv;
  }
  q = wave_sum(q);
  if (lane == 0) red[wv] = q;
  __syncthreads();
  if (tid == 0) {
    float num = 0.f;
    for (int j = 0; j < 16; ++j) num += red[j];
    const float den = ub * ub + eps;
    sc[0] = ub;
    sc[1] = num;
    sc[2] = den;
    if (loss) *loss = num / den;
  }
}

// A workgroup per row e:
//   du_c = 2 (u_c - ub) / den - num 2 ub / (C den^2),
//   dL[e][c] = lambda / R p_ec (du_c - sum_c' p_ec' du_c') + dw[e][i] where c = s_ei.
__global__ void __launch_bounds__(kBwThreads)
k_cov_grad(const float* __restrict__ L, const float* __restrict__ mz, const float* __restrict__ u,
           const float* __restrict__ sc, const int32_t* __restrict__ s, const float* __restrict__ dw,
           float* __restrict__ dL, int R, int C, int k, float lambda) {
  extern __shared__ int32_t pos[];  // [C]: support position of channel c in this row, or -1
  __shared__ float red[kBwWaves];
  const int e = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float* row = L + (int64_t)e * C;
  const float m = mz[2 * e], rz = 1.f / mz[2 * e + 1];
  const float ub = sc[0], num = sc[1], den = sc[2];
  const float c1 = 2.f / den, c0 = num * 2.f * ub / ((float)C * den * den);
  if (dw) {
    for (int c = tid; c < C; c += kBwThreads) pos[c] = -1;
    __syncthreads();
    for (int i = tid; i < k; i += kBwThreads) pos[s[(int64_t)e * k + i]] = i;
  }
  float t = 0.f;
  for (int c = tid; c < C; c += kBwThreads) {
    const float p = expf(row[c] - m) * rz;
    t += p * (c1 * (u[c] - ub) - c0);
  }
  t = wave_sum(t);
  if (lane == 0) red[wv] = t;
  __syncthreads();
  float tt = 0.f;
  for (int j = 0; j < kBwWaves; ++j) tt += red[j];
  const float scale = lambda / (float)R;
  for (int c = tid; c < C; c += kBwThreads) {
    const float p = expf(row[c] - m) * rz;
    float g = scale * p * ((c1 * (u[c] - ub) - c0) - tt);
    if (dw) {
      const int i = pos[c];
      if (i >= 0) g += dw[(int64_t)e * k + i];
    }
    dL[(int64_t)e * C + c] = g;
  }
}

unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

// image groups of the sums over images: about 2048 workgroups, at most 64
// groups
void backward_sum_groups(const Shape& sh, int* ng, int* gs) {
  const int64_t blocks = std::max<int64_t>(1, ((int64_t)sh.R * sh.k + kBwThreads - 1) / kBwThreads);
  const int64_t want = std::max<int64_t>(1, std::min<int64_t>({sh.B, (int64_t)64, (2048 + blocks - 1) / blocks}));
  *gs = (int)((sh.B + want - 1) / want);
  *ng = (int)((sh.B + *gs - 1) / *gs);
}

bool backward_supported(const Shape& sh, int gate_kind) {
  return sh.k <= kBwMaxK && (gate_kind != MOCE_GATE_MLP_SIGMOID || sh.k <= kMlpBwMaxK);
}

size_t backward_mlp_parts(const Shape& sh) {
  const int64_t nblk = (sh.B * sh.R + kMlpBwRows - 1) / kMlpBwRows;
  return (size_t)std::max<int64_t>(1, std::min<int64_t>(nblk, 512));
}

size_t backward_mlp_part_floats(const Shape& sh) { return (size_t)sh.k * sh.k + 2 * (size_t)sh.k + 1; }

hipError_t launch_backward(const Shape& sh, const void* x, const void* dy, const int32_t* s, const float* w,
                           const moce_gate_params& g, void* dx, float* dw, const moce_gate_grads& gg,
                           const BwdWs& ws, hipStream_t st) {
  const int64_t B = sh.B, HW = sh.HW;
  const int C = (int)sh.C, E = sh.E, R = sh.R, k = sh.k;
  const bool bf = sh.elem == MOCE_BF16, nhwc = sh.layout == MOCE_NHWC;
  const bool mlp = g.kind == MOCE_GATE_MLP_SIGMOID;
  hipError_t err;
  // inverse support map (also |U|)
  k_bw_fill_i32<<<blocks_for(C + 1, 256), 256, 0, st>>>(ws.cnt, C + 1, 0);
  if (R > 0) {
    const int64_t n = (int64_t)R * k;
    k_inv_count<<<blocks_for(n, 256), 256, 0, st>>>(s, n, ws.cnt);
  }
  k_inv_scan<<<1, 1024, 0, st>>>(ws.cnt, ws.off, ws.cur, ws.nU, C);
  if (R > 0) {
    const int64_t n = (int64_t)R * k;
    k_inv_fill<<<blocks_for(n, 256), 256, 0, st>>>(s, n, ws.cur, ws.inv);
    k_inv_sort<<<blocks_for(C, 4), 256, 0, st>>>(ws.off, ws.inv, C);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    // forward quantities: d, the softmax statistics and the coefficients
    if ((err = launch_pool(sh, x, ws.d, st)) != hipSuccess) return err;
    // the coefficients themselves only for the generic dx (the matrix-core dx
    // rebuilds them from the statistics)
    int nbk;
    int64_t nem;
    bwd_dx_sched_sizes(sh, &nbk, &nem);
    float* alpha_out = nbk > 0 ? nullptr : ws.alpha;
    if ((err = launch_gate(sh, ws.d, s, w, g, ws.tau, alpha_out, ws.stats, st)) != hipSuccess) return err;
    // dalpha
    if (!bwd_mfma_dalpha(sh, x, dy, s, ws, st, &err)) {
      const unsigned nb = blocks_for(B * R, kBwWaves);
      if (bf) {
        auto xx = static_cast<const uint16_t*>(x);
        auto gy = static_cast<const uint16_t*>(dy);
        if (nhwc)
          k_bw_dalpha<uint16_t, true><<<nb, kBwThreads, 0, st>>>(xx, gy, s, ws.dal, B, C, E, R, k, (int)HW);
        else
          k_bw_dalpha<uint16_t, false><<<nb, kBwThreads, 0, st>>>(xx, gy, s, ws.dal, B, C, E, R, k, (int)HW);
      } else {
        auto xx = static_cast<const float*>(x);
        auto gy = static_cast<const float*>(dy);
        if (nhwc)
          k_bw_dalpha<float, true><<<nb, kBwThreads, 0, st>>>(xx, gy, s, ws.dal, B, C, E, R, k, (int)HW);
        else
          k_bw_dalpha<float, false><<<nb, kBwThreads, 0, st>>>(xx, gy, s, ws.dal, B, C, E, R, k, (int)HW);
      }
      err = hipGetLastError();
    }
    if (err != hipSuccess) return err;
    // rows
    {
      int nsplit = 1, split_len = 0;
      bwd_dalpha_splits(sh, &nsplit, &split_len);
      const unsigned nb = blocks_for(B * R, kBwWaves);
      const float* a = mlp ? nullptr : g.a;
      const float* cc = mlp ? nullptr : g.c;
      const int npl = (k + kWave - 1) / kWave;
#define MOCE_BW_ROWS(N) \
  k_bw_rows<N><<<nb, kBwThreads, 0, st>>>(ws.dal, w, ws.stats, ws.d, s, a, cc, ws.S1, ws.dtau, ws.dg, B, C, R, k, \
                                          nsplit)
      if (npl <= 1)
        MOCE_BW_ROWS(1);
      else if (npl <= 2)
        MOCE_BW_ROWS(2);
      else if (npl <= 4)
        MOCE_BW_ROWS(4);
      else if (npl <= 8)
        MOCE_BW_ROWS(8);
      else
        MOCE_BW_ROWS(16);
#undef MOCE_BW_ROWS
      if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    if (mlp) {
      const int nparts = (int)backward_mlp_parts(sh);
      const size_t lds = ((size_t)k * k + 2 * (size_t)kMlpBwRows * k + kMlpBwRows) * sizeof(float);
      if (lds > 64 * 1024 &&
          (err = hipFuncSetAttribute((const void*)k_bw_mlp, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) !=
              hipSuccess)
        return err;
      k_bw_mlp<<<nparts, kBwThreads, lds, st>>>(ws.d, s, ws.dtau, g.W1, g.b1, g.w2, g.b2, g.tau_min, g.tau_max,
                                                 ws.dzg, ws.part, B, C, R, k);
      const int nq = (int)backward_mlp_part_floats(sh);
      k_bw_mlp_reduce<<<blocks_for(nq, 256), 256, 0, st>>>(ws.part, nparts, k, gg.dW1, gg.db1, gg.dw2, gg.db2);
      if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    {
      int ng, gs;
      backward_sum_groups(sh, &ng, &gs);
      const int64_t rk = (int64_t)R * k;
      k_bw_sums<<<dim3(blocks_for(rk, kBwThreads), ng), kBwThreads, 0, st>>>(
          ws.dal, w, ws.stats, ws.S1, ws.dg, ws.d, s, ws.psum, ws.psum + ng * rk, ws.psum + 2 * ng * rk, B, C, R, k,
          gs, !mlp);
      k_bw_sums_reduce<<<blocks_for(std::max<int64_t>(rk, R), 256), 256, 0, st>>>(
          ws.psum, ws.psum + ng * rk, ws.psum + 2 * ng * rk, ng, rk, R, dw, mlp ? nullptr : gg.da,
          mlp ? nullptr : gg.dc);
    }
    k_bw_dd<<<blocks_for(B * C, kBwThreads), kBwThreads, 0, st>>>(ws.off, ws.inv, ws.dg, mlp ? nullptr : g.a,
                                                                   ws.dzg, ws.dd, B, C, R, k);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  // dx
  if (bwd_mfma_dx(sh, dy, s, w, ws, dx, st, &err)) return err;
  const unsigned nb = blocks_for(B * C * HW, kBwThreads);
  if (bf) {
    auto gy = static_cast<const uint16_t*>(dy);
    auto o = static_cast<uint16_t*>(dx);
    if (nhwc)
      k_bw_dx<uint16_t, true><<<nb, kBwThreads, 0, st>>>(gy, ws.alpha, ws.off, ws.inv, ws.nU, ws.dd, o, B, C, E, R,
                                                         k, (int)HW);
    else
      k_bw_dx<uint16_t, false><<<nb, kBwThreads, 0, st>>>(gy, ws.alpha, ws.off, ws.inv, ws.nU, ws.dd, o, B, C, E,
                                                          R, k, (int)HW);
  } else {
    auto gy = static_cast<const float*>(dy);
    auto o = static_cast<float*>(dx);
    if (nhwc)
      k_bw_dx<float, true><<<nb, kBwThreads, 0, st>>>(gy, ws.alpha, ws.off, ws.inv, ws.nU, ws.dd, o, B, C, E, R, k,
                                                      (int)HW);
    else
      k_bw_dx<float, false><<<nb, kBwThreads, 0, st>>>(gy, ws.alpha, ws.off, ws.inv, ws.nU, ws.dd, o, B, C, E, R,
                                                       k, (int)HW);
  }
  return hipGetLastError();
}

bool logit_backward_supported(int64_t C) { return C >= 1 && C <= kCovMaxC; }

hipError_t launch_logit_backward(int R, int C, int k, const float* L, const int32_t* s, const float* dw, float eps,
                                 float lambda, float* loss, float* dL, float* ws, hipStream_t st) {
  float* mz = ws;                 // [2 R]
  float* u = mz + 2 * (size_t)R;  // [C]
  float* sc = u + C;              // [3]
  const size_t lds = dw ? (size_t)C * sizeof(int32_t) : 0;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_cov_grad, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  k_cov_rows<<<R, kBwThreads, 0, st>>>(L, mz, C);
  k_cov_cols<<<blocks_for(C, 256), 256, 0, st>>>(L, mz, u, R, C);
  k_cov_scalar<<<1, 1024, 0, st>>>(u, C, eps, sc, loss);
  k_cov_grad<<<R, kBwThreads, lds, st>>>(L, mz, u, sc, s, dw, dL, R, C, k, lambda);
  return hipGetLastError();
}

}  // namespace moce

// Mixing as a dense product on the matrix cores (gfx950 MFMA).
//
// For one image b the routed outputs (Sec. 3.3 Eq. 5) and the residual output
// (Sec. 3.4 Eq. 6) are a single linear map of the channels:
//   y[b][o][p] = sum_c A_b[o][c] x[b][c][p],
// where row o < E-1 of A_b holds alpha[b][o][i] at column s[o][i] and row E-1
// holds 1/|U| at the uncovered channels (zero when U is empty).  A_b has k of
// C entries per row (1/8 for the ResNet-50 stage-1 layer), but the matrix
// cores multiply a dense bf16 tile far faster than the vector ALUs run the
// gather-and-FMA form, so the kernel builds A_b densely and evaluates
// y^T = x^T A_b^T with 32x32x16 bf16 MFMAs, which leaves it bound by HBM.
//
// Exactness.  x is bf16 already.  Each float32 coefficient is split into bf16
// parts hi + mid + lo that sum to it exactly, one MFMA per part: bf16 x bf16
// products are exact in float32 and the MFMA accumulates in float32, so the
// result is the float32 gather form up to the order of the additions.
//
// Work split.  A workgroup of 4 waves occupies one CU and walks a contiguous
// range of tiles (64 positions x all C channels of one image).  Wave w
// computes positions 32 (w & 1) .. +31 of the tile for experts 32 (w >> 1) ..
// +31.  Each wave holds its 32 rows of A_b (all channels, every part) in
// registers as MFMA B operands, rebuilt when the image changes; the x tile is
// held in LDS as bf16 and read as MFMA A operands with the transposing LDS
// read, which turns the position-contiguous rows into channel-contiguous
// operands.  Three tiles are in flight in registers while one is multiplied.
#include <algorithm>

#include "moce_internal.h"

namespace moce {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#define MOCE_LDS __attribute__((address_space(3)))

constexpr int kThreads = 256;
constexpr int kTile = 64;          // positions per tile
constexpr int kRow = kTile * 2;    // bytes of one channel row of an LDS tile
constexpr int kMaxE = 64;          // rows of A_b
constexpr int kMaxC = 256;
constexpr int kPre = 8;            // coefficient entries per thread fetched into registers

struct MixArgs {
  int C, HW, E, R, k, nU, nt, ntiles;
};

// LDS: two x tiles [C][kTile] bf16, then the staging rows of A_b
// [kMaxE][C + 8] bf16 (the 8-element pad spreads the rows over the banks).
__host__ __device__ inline int stage_row(int C) { return C + 8; }
__host__ __device__ inline size_t mfma_lds(int C) {
  return (size_t)2 * C * kRow + (size_t)kMaxE * stage_row(C) * 2;
}

// Chunk q (16 bytes = 8 positions) of channel row c is stored at chunk
// q ^ swz(c), so that the 8 rows x 64 bytes one transposing read touches
// fall evenly on the LDS banks.
__device__ __forceinline__ int swz(int c) { return ((c >> 1) & 1) << 2; }

// Global loads of tile n (NR rounds of 16 bytes per thread): thread t reads
// positions 8 (t & 7) .. +7 of channel (t >> 3) + 32 u.  Positions past the
// image repeat its last vector; those outputs are never stored.
template <int NR>
__device__ __forceinline__ void load_tile(const MixArgs& p, const uint16_t* __restrict__ x, int n, u32x4 (&buf)[NR],
                                          int tid) {
  const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
  const int p0 = j * kTile;
  const int vq = min(tid & 7, min(kTile, p.HW - p0) / 8 - 1);
  const uint16_t* src = x + ((int64_t)b * p.C + (tid >> 3)) * p.HW + p0 + vq * 8;
#pragma unroll
  for (int u = 0; u < NR; ++u) buf[u] = *reinterpret_cast<const u32x4*>(src + (int64_t)u * 32 * p.HW);
}

template <int NR>
__device__ __forceinline__ void store_tile(const u32x4 (&buf)[NR], unsigned char* dst, int tid) {
  const int c = tid >> 3, q = tid & 7;
  unsigned char* d = dst + c * kRow + ((q ^ swz(c)) << 4);
#pragma unroll
  for (int u = 0; u < NR; ++u) *reinterpret_cast<u32x4*>(d + u * 32 * kRow) = buf[u];
}

// Part `part` of the exact split a = hi + mid + lo into bf16 values (with
// two parts: hi and the rounded remainder).
__device__ __forceinline__ uint16_t coef_part(float a, int part) {
  const uint16_t hi = f32_to_bf16(a);
  if (part == 0) return hi;
  const float r1 = a - bf16_to_f32(hi);
  const uint16_t mid = f32_to_bf16(r1);
  if (part == 1) return mid;
  return f32_to_bf16(r1 - bf16_to_f32(mid));
}

// Coefficients of one image fetched into registers ahead of the rebuild:
// entry e = tid + 256 r of alpha[b] (the flattened [R][k] block).
struct CoefFetch {
  float a[kPre];
};

__device__ __forceinline__ void fetch_coefs(const MixArgs& p, const float* __restrict__ alpha, int b, CoefFetch& f,
                                            int tid) {
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
#pragma unroll
  for (int r = 0; r < kPre; ++r) f.a[r] = ab[min(tid + kThreads * r, nent - 1)];
}

// Rebuilds the wave's rows of A_b in registers: zero the staging rows, then
// per part scatter the coefficients (and 1/nU at the uncovered channels) and
// read the MFMA B operands.  slot[r] is the staging index of entry
// tid + 256 r; entries past kPre * 256 are read here directly.
template <int NS, int NKS>
__device__ __forceinline__ void build_coefs(const MixArgs& p, int b, const int32_t* __restrict__ s, const float* __restrict__ alpha,
                            int uch, const CoefFetch& f, const int (&slot)[kPre], uint16_t* stage,
                            bf16x8 (&bfr)[NS][NKS], int tid, int orow, int khalf) {
  const int rs = stage_row(p.C);
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
  const float inv = p.nU > 0 ? 1.f / (float)p.nU : 0.f;
  uint4* z = reinterpret_cast<uint4*>(stage);
  const int nz = kMaxE * rs / 8;
  for (int i = tid; i < nz; i += kThreads) z[i] = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
  for (int part = 0; part < NS; ++part) {
    __syncthreads();  // zeroing (or the previous part's operand reads) done
#pragma unroll
    for (int r = 0; r < kPre; ++r)
      if (tid + kThreads * r < nent) stage[slot[r]] = coef_part(f.a[r], part);
    for (int e = tid + kThreads * kPre; e < nent; e += kThreads)
      stage[(e / p.k) * rs + s[e]] = coef_part(ab[e], part);
    if (tid < p.nU) stage[p.R * rs + uch] = coef_part(inv, part);
    __syncthreads();
    const uint16_t* row = stage + orow * rs + khalf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      bfr[part][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(row + ks * 16));
  }
}

__device__ __forceinline__ bf16x4 tr_read(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MOCE_LDS bf16x4*)(MOCE_LDS unsigned char*)p);
}

// NR = C / 32 load rounds, NS coefficient parts.
template <int NR, int NS>
__global__ void __launch_bounds__(kThreads, 1)
k_mfmamix(MixArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, const int32_t* __restrict__ s,
          const float* __restrict__ alpha, const int32_t* __restrict__ U) {
  constexpr int NKS = 2 * NR;  // channel steps of 16
  extern __shared__ __align__(16) unsigned char smem[];
  const int G = gridDim.x;
  const int t0 = (int)((int64_t)blockIdx.x * p.ntiles / G);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * p.ntiles / G);
  if (t0 >= t1) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mb = wv & 1, nb = wv >> 1;
  const int tileb = p.C * kRow;
  uint16_t* stage = reinterpret_cast<uint16_t*>(smem + 2 * tileb);
  const int rs = stage_row(p.C);

  // coefficients and static scatter slots first, so that waiting for them
  // does not wait for the tiles
  int cur = t0 / p.nt;
  CoefFetch f;
  fetch_coefs(p, alpha, cur, f, tid);
  int slot[kPre];
  const int nent = p.R * p.k;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const int e = min(tid + kThreads * r, nent - 1);
    slot[r] = (e / p.k) * rs + s[e];
  }
  // uncovered channel tid (U may be null when nU == 0: s is read instead)
  const int uv = *(p.nU > 0 ? U + min(tid, p.nU - 1) : s);
  const int uch = p.nU > 0 ? uv : 0;

  u32x4 st0[NR], st1[NR], st2[NR];
  // issue order t0, t0 + 1, t0 + 2 (the loop below relies on loads
  // completing in that order)
  load_tile(p, x, t0, st0, tid);
  __builtin_amdgcn_sched_barrier(0);
  load_tile(p, x, min(t0 + 1, t1 - 1), st1, tid);
  __builtin_amdgcn_sched_barrier(0);
  load_tile(p, x, min(t0 + 2, t1 - 1), st2, tid);
  __builtin_amdgcn_sched_barrier(0);

  bf16x8 bfr[NS][NKS];
  build_coefs<NS, NKS>(p, cur, s, alpha, uch, f, slot, stage, bfr, tid, 32 * nb + (lane & 31), lane >> 5);
  store_tile(st0, smem, tid);
  __syncthreads();

  // transposing-read offset of this lane for channel step 0, first half:
  // 16-lane group g reads channels 8 (g >> 1) + 4 h + (l >> 2) at positions
  // 32 mb + 16 (g & 1) + 4 (l & 3) .. +3 (l = lane & 15)
  const int g = lane >> 4, sl = lane & 15;
  const int trow = 8 * (g >> 1) + (sl >> 2);
  const int tq = 4 * mb + 2 * (g & 1) + ((sl & 3) >> 1);
  const int troff = trow * kRow + ((tq ^ (((sl >> 3) & 1) << 2)) << 4) + 8 * (sl & 1);
  const int o = 32 * nb + (lane & 31);

  auto step = [&](int n, u32x4(&refill)[NR], const u32x4(&next)[NR]) __attribute__((always_inline)) {
    const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
    if (b != cur) {
      build_coefs<NS, NKS>(p, b, s, alpha, uch, f, slot, stage, bfr, tid, 32 * nb + (lane & 31), lane >> 5);
      cur = b;
    }
    const int n1 = n + 1;
    if (n1 < t1 && n1 / p.nt != b) fetch_coefs(p, alpha, n1 / p.nt, f, tid);
    load_tile(p, x, min(n + 3, t1 - 1), refill, tid);
    __builtin_amdgcn_sched_barrier(0);  // the loads go out before the products

    const unsigned char* tb = smem + ((n - t0) & 1) * tileb + troff;
    bf16x8 xa[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x4 lo = tr_read(tb + ks * 16 * kRow);
      const bf16x4 hi = tr_read(tb + ks * 16 * kRow + 4 * kRow);
      xa[ks] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    f32x16 acc0 = {}, acc1 = {};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int part = 0; part < NS; ++part) {
        if (((ks * NS + part) & 1) == 0)
          acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[ks], bfr[part][ks], acc0, 0, 0, 0);
        else
          acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[ks], bfr[part][ks], acc1, 0, 0, 0);
      }

    // the next tile into the other buffer (its last readers passed the
    // barrier that ended the previous step)
    store_tile(next, smem + ((n - t0 + 1) & 1) * tileb, tid);

    // lane holds expert o at positions 32 mb + 8 q + 4 (lane >> 5) .. +3
    const int pb = j * kTile + 32 * mb + 4 * (lane >> 5);
    uint16_t* yo = y + ((int64_t)b * p.E + o) * p.HW + pb;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float v0 = acc0[4 * q] + acc1[4 * q], v1 = acc0[4 * q + 1] + acc1[4 * q + 1];
      const float v2 = acc0[4 * q + 2] + acc1[4 * q + 2], v3 = acc0[4 * q + 3] + acc1[4 * q + 3];
      if (o < p.E && pb + 8 * q < p.HW)
        *reinterpret_cast<uint2*>(yo + 8 * q) = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
    }
    __syncthreads();
  };

  for (int n = t0;;) {
    step(n, st0, st1);
    if (++n >= t1) break;
    step(n, st1, st2);
    if (++n >= t1) break;
    step(n, st2, st0);
    if (++n >= t1) break;
  }
}

using MfmaKernel = void (*)(MixArgs, const uint16_t*, uint16_t*, const int32_t*, const float*, const int32_t*);

template <int NS>
MfmaKernel pick(int nr) {
  static const MfmaKernel k[8] = {k_mfmamix<1, NS>, k_mfmamix<2, NS>, k_mfmamix<3, NS>, k_mfmamix<4, NS>,
                                  k_mfmamix<5, NS>, k_mfmamix<6, NS>, k_mfmamix<7, NS>, k_mfmamix<8, NS>};
  return k[nr - 1];
}

constexpr int kParts = 3;

}  // namespace

bool mfmamix_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.C % 32 != 0 || sh.C > kMaxC || sh.E > kMaxE || sh.HW % 8 != 0) return false;
  const int64_t nt = (sh.HW + kTile - 1) / kTile;
  if (sh.B * nt > INT32_MAX / 2) return false;
  return true;
}

hipError_t launch_mfmamix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st) {
  MixArgs p;
  p.C = (int)sh.C;
  p.HW = (int)sh.HW;
  p.E = sh.E;
  p.R = sh.R;
  p.k = sh.k;
  p.nU = nU;
  p.nt = (int)((sh.HW + kTile - 1) / kTile);
  p.ntiles = (int)(sh.B * p.nt);
  if (p.ntiles == 0) return hipSuccess;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  const int grid = std::min(cus, p.ntiles);
  const size_t lds = mfma_lds(p.C);
  const MfmaKernel k = pick<kParts>(p.C / 32);
  static bool configured[8] = {};
  if (!configured[p.C / 32 - 1]) {
    const hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    configured[p.C / 32 - 1] = true;
  }
  hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, st, p, static_cast<const uint16_t*>(x),
                     static_cast<uint16_t*>(y), s, alpha, U);
  return hipGetLastError();
}

}  // namespace moce

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
// y^T = x^T A_b^T with 16x16x32 bf16 MFMAs, which leaves it bound by memory.
//
// Exactness.  x is bf16 already.  Each float32 coefficient is split into bf16
// parts hi + mid + lo that sum to it exactly, one MFMA per part: bf16 x bf16
// products are exact in float32 and the MFMA accumulates in float32, so the
// result is the float32 gather form up to the order of the additions.
//
// Work split.  Two workgroups of 4 waves share a CU, so that one multiplies
// while the other loads, stores and synchronises.  A workgroup walks a
// contiguous range of tiles (64 positions x all C channels of one image);
// wave w computes experts 16 w .. 16 w + 15 at all 64 positions.  Each wave
// holds its 16 rows of A_b (all channels, every part) in registers as MFMA B
// operands, rebuilt when the image changes.  The x tile is held in LDS as
// bf16, double-buffered, and read as MFMA A operands with the transposing LDS
// read, which turns position-contiguous channel rows into channel-contiguous
// operands.  A_b is assembled in whichever tile buffer is free at that moment.
// Results leave through a small per-wave LDS area so that every store
// instruction writes whole 128-byte rows of y.
#include <algorithm>
#include <type_traits>

#include "moce_internal.h"

namespace moce {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
#define MOCE_LDS __attribute__((address_space(3)))

constexpr int kThreads = 256;
constexpr int kTile = 64;               // positions per tile
constexpr int kRow = kTile * 2;         // bytes of one channel row of an LDS tile
constexpr int kMaxE = 64;               // rows of A_b
constexpr int kMaxC = 256;
constexpr int kPre = 8;                 // coefficient entries per thread fetched into registers
constexpr int kExpertsPerWave = 16;
constexpr int kOutRow = kRow + 16;      // bytes per row of a wave's output area (padded)
constexpr int kOutWave = kExpertsPerWave * kOutRow;
// s_waitcnt operand waiting for every vector memory access (vmcnt 0, the
// LDS/scalar and export counters left at their maxima)
constexpr int kVmDrain = 0x0f70;

struct MixArgs {
  int C, HW, E, R, k, nU, nt, ntiles;
};

// LDS: two x tiles [C][kTile] bf16, then the four waves' output areas.
__host__ __device__ inline size_t mfma_lds(int C) { return (size_t)2 * C * kRow + (size_t)4 * kOutWave; }

// Chunk q (16 bytes = 8 positions) of channel row c of a tile is stored at
// chunk q ^ (2 ((c >> 3) & 3)): the 16 rows x 32 bytes that one transposing
// read touches then fall on the LDS banks two deep, the least possible.
__device__ __forceinline__ int tile_swz(int c) { return ((c >> 3) & 3) << 1; }

// Byte offset of A_b[o][c] in the staging area [kMaxE][C] bf16, whose 16-byte
// chunks are rotated by 4 (o & 3) within the row so that the operand reads
// (16 rows x 64 bytes) spread over the banks.
__device__ __forceinline__ int stage_off(int o, int c, int C) {
  const int nch = C >> 3;
  int ch = (c >> 3) + 4 * (o & 3);
  ch = ch >= nch ? ch - nch : ch;
  ch = ch >= nch ? ch - nch : ch;
  ch = ch >= nch ? ch - nch : ch;
  return o * C * 2 + ch * 16 + (c & 7) * 2;
}

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

// Thread t's chunks go to rows (t >> 3) + 32 u: one wave writes 8 whole rows.
template <int NR>
__device__ __forceinline__ void store_tile(const u32x4 (&buf)[NR], unsigned char* dst, int tid) {
  const int c = tid >> 3, q = tid & 7;
  unsigned char* d = dst + c * kRow + ((q ^ tile_swz(c)) << 4);
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

// Entries tid + 256 r of alpha[b] (the flattened [R][k] block), fetched
// ahead of a rebuild.
__device__ __forceinline__ void fetch_coefs(const MixArgs& p, const float* __restrict__ alpha, int b,
                                            float (&a)[kPre], int tid) {
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
#pragma unroll
  for (int r = 0; r < kPre; ++r) a[r] = ab[min(tid + kThreads * r, nent - 1)];
}

// Rebuilds the wave's rows of A_b in registers, assembling A_b in the tile
// buffer `stage` (free while this runs): zero it, then per part scatter the
// coefficients alpha[b] (a: the first kPre * 256 of them, fetched ahead; the
// rest are read here) and 1/nU at the uncovered channels, and read the MFMA B
// operands.  The staging offset of entry e = tid + 256 r (below 2^15) is the
// 16-bit half r & 1 of slot[r >> 1].  Ends with a barrier, after which the
// buffer may be overwritten.
template <int NS, int NR>
__device__ __forceinline__ void build_coefs(const MixArgs& p, int b, const int32_t* __restrict__ s,
                                            const float* __restrict__ alpha, const float (&a)[kPre], int uch,
                                            const uint32_t (&slot)[kPre / 2], unsigned char* stage,
                                            bf16x8 (&bfr)[NS][NR], int tid, int orow, int kq) {
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
  const float inv = p.nU > 0 ? 1.f / (float)p.nU : 0.f;
  u32x4* z = reinterpret_cast<u32x4*>(stage);
  const int nz = kMaxE * p.C / 8;
  for (int i = tid; i < nz; i += kThreads) z[i] = u32x4{0u, 0u, 0u, 0u};
  const int ures = stage_off(p.R, uch, p.C);
#pragma unroll
  for (int part = 0; part < NS; ++part) {
    __syncthreads();  // zeroing (or the previous part's operand reads) done
#pragma unroll
    for (int r = 0; r < kPre; ++r)
      if (tid + kThreads * r < nent)
        *reinterpret_cast<uint16_t*>(stage + ((slot[r >> 1] >> (16 * (r & 1))) & 0xffffu)) = coef_part(a[r], part);
    for (int e = tid + kThreads * kPre; e < nent; e += kThreads)
      *reinterpret_cast<uint16_t*>(stage + stage_off(e / p.k, s[e], p.C)) = coef_part(ab[e], part);
    if (tid < p.nU) *reinterpret_cast<uint16_t*>(stage + ures) = coef_part(inv, part);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < NR; ++ks)
      bfr[part][ks] =
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(stage + stage_off(orow, 32 * ks + 8 * kq, p.C)));
  }
  __syncthreads();
}

__device__ __forceinline__ bf16x4 tr_read(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MOCE_LDS bf16x4*)(MOCE_LDS unsigned char*)p);
}

// NR = C / 32 load rounds (and channel steps of 32), NS coefficient parts.
template <int NR, int NS>
__global__ void __launch_bounds__(kThreads, 2)
k_mfmamix(MixArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, const int32_t* __restrict__ s,
          const float* __restrict__ alpha, const int32_t* __restrict__ U) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int G = gridDim.x;
  const int t0 = (int)((int64_t)blockIdx.x * p.ntiles / G);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * p.ntiles / G);
  if (t0 >= t1) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tileb = p.C * kRow;
  unsigned char* outw = smem + 2 * tileb + wv * kOutWave;
  const int orow = kExpertsPerWave * wv + (lane & 15);  // this lane's expert (operand row, output column)
  const int g = lane >> 4, sl = lane & 15;

  // static scatter offsets, the uncovered channel and the first image's
  // coefficients are read before any tile is requested (every workgroup
  // starting at once would otherwise queue these small reads behind
  // megabytes of tile requests); the first rebuild then runs while tile t0
  // is in flight
  uint32_t slot[kPre / 2] = {};
  const int nent = p.R * p.k;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const int e = min(tid + kThreads * r, nent - 1);
    slot[r >> 1] |= (uint32_t)stage_off(e / p.k, s[e], p.C) << (16 * (r & 1));
  }
  // uncovered channel tid (U may be null when nU == 0: s is read instead)
  const int uv = *(p.nU > 0 ? U + min(tid, p.nU - 1) : s);
  const int uch = p.nU > 0 ? uv : 0;
  int b = t0 / p.nt, j = t0 - b * p.nt;
  float a[kPre];
  fetch_coefs(p, alpha, b, a, tid);
  __builtin_amdgcn_s_waitcnt(kVmDrain);
  __builtin_amdgcn_sched_barrier(0);

  // issue order t0, t0 + 1 (the loop below relies on loads completing in
  // that order)
  u32x4 st0[NR], st1[NR];
  load_tile(p, x, t0, st0, tid);
  __builtin_amdgcn_sched_barrier(0);
  bf16x8 bfr[NS][NR];
  build_coefs<NS, NR>(p, b, s, alpha, a, uch, slot, smem + tileb, bfr, tid, orow, g);
  __builtin_amdgcn_sched_barrier(0);
  load_tile(p, x, min(t0 + 1, t1 - 1), st1, tid);
  __builtin_amdgcn_sched_barrier(0);
  store_tile(st0, smem, tid);  // tile t0 into buffer 0
  __syncthreads();

  // transposing reads: 16-lane group g reads channels 8 g + 4 h + (l >> 2)
  // (+ 32 ks) at positions 16 pb + 4 (l & 3) .. +3, l = lane & 15
  const int trow = (8 * g + (sl >> 2)) * kRow + 8 * (sl & 1);
  int troff[4];
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) troff[pb] = trow + (((2 * pb + ((sl & 3) >> 1)) ^ (2 * g)) << 4);
  // this thread's destination of tile rows (tid >> 3) + 32 u
  const int stoff = (tid >> 3) * kRow + (((tid & 7) ^ tile_swz(tid >> 3)) << 4);

  // results of the previous tile, bf16: expert orow at positions 16 pb + 4 g
  // .. +3 of tile (pb_img, pj); written through the wave's output area so
  // that lane i stores 16 bytes of row i >> 3 (+8)
  u32x2 prev[4];
  int pb_img = b, pj = j;
  auto emit = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) *reinterpret_cast<u32x2*>(outw + sl * kOutRow + 32 * pb + 8 * g) = prev[pb];
    const int pos = pj * kTile + 8 * (lane & 7);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = (lane >> 3) + 8 * h;
      const u32x4 v = *reinterpret_cast<const u32x4*>(outw + r * kOutRow + (lane & 7) * 16);
      const int o = kExpertsPerWave * wv + r;
      if (o < p.E && pos < p.HW) *reinterpret_cast<u32x4*>(y + ((int64_t)pb_img * p.E + o) * p.HW + pos) = v;
    }
  };

  // Tile n: the previous tile's results leave, tile n + 2 is requested into
  // the registers tile n came through, and the products of tile n run with
  // tile n + 1 written into the other buffer a row chunk per channel step
  // (waiting for tile n + 1 only).  The other buffer is free: the barrier
  // that ended the previous step (or the rebuild) follows the last reads of
  // tile n - 1.
  auto step = [&](int n, auto first, u32x4(&refill)[NR], const u32x4(&next)[NR]) __attribute__((always_inline)) {
    if constexpr (!decltype(first)::value) emit();
    load_tile(p, x, min(n + 2, t1 - 1), refill, tid);
    unsigned char* other = smem + ((n - t0 + 1) & 1) * tileb + stoff;
    const unsigned char* tb = smem + ((n - t0) & 1) * tileb;
    f32x4 acc[4];
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) acc[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NR; ++ks) {
#pragma unroll
      for (int pb = 0; pb < 4; ++pb) {
        const unsigned char* ap = tb + troff[pb] + ks * 32 * kRow;
        const bf16x8 xa = __builtin_shufflevector(tr_read(ap), tr_read(ap + 4 * kRow), 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int part = 0; part < NS; ++part)
          acc[pb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa, bfr[part][ks], acc[pb], 0, 0, 0);
      }
      *reinterpret_cast<u32x4*>(other + ks * 32 * kRow) = next[ks];
    }
#pragma unroll
    for (int pb = 0; pb < 4; ++pb)
      prev[pb] = u32x2{pack_bf16x2(acc[pb][0], acc[pb][1]), pack_bf16x2(acc[pb][2], acc[pb][3])};
    pb_img = b;
    pj = j;
    __syncthreads();  // tile n + 1 visible; every read of tile n done
  };

  // tiles t0 + 1 ..: one image at a time, A_b rebuilt unconditionally at the
  // start of each image's run, so that the operand registers are never merged
  // across a conditional rebuild
  auto run = [&](int n, int te) __attribute__((always_inline)) {
#pragma unroll 2
    for (; n < te; ++n, ++j) {
      step(n, std::false_type{}, st0, st1);
      // tile n + 2 now sits in st0 and tile n + 1 has left st1
      u32x4 sw[NR];
#pragma unroll
      for (int u = 0; u < NR; ++u) sw[u] = st0[u];
#pragma unroll
      for (int u = 0; u < NR; ++u) st0[u] = st1[u];
#pragma unroll
      for (int u = 0; u < NR; ++u) st1[u] = sw[u];
    }
  };

  step(t0, std::true_type{}, st0, st1);
  {
    u32x4 sw[NR];
#pragma unroll
    for (int u = 0; u < NR; ++u) sw[u] = st0[u];
#pragma unroll
    for (int u = 0; u < NR; ++u) st0[u] = st1[u];
#pragma unroll
    for (int u = 0; u < NR; ++u) st1[u] = sw[u];
  }
  ++j;
  int n = t0 + 1;
  run(n, min(t1, (b + 1) * p.nt));
  n = min(t1, (b + 1) * p.nt);
  while (n < t1) {
    // next image: this workgroup stalls on the coefficient loads, the other
    // one on the CU keeps it busy
    ++b;
    j = 0;
    fetch_coefs(p, alpha, b, a, tid);
    build_coefs<NS, NR>(p, b, s, alpha, a, uch, slot, smem + ((n - t0 + 1) & 1) * tileb, bfr, tid, orow, g);
    const int te = min(t1, (b + 1) * p.nt);
    run(n, te);
    n = te;
  }
  emit();
}

using MfmaKernel = void (*)(MixArgs, const uint16_t*, uint16_t*, const int32_t*, const float*, const int32_t*);

template <int NS>
MfmaKernel pick(int nr) {
  static const MfmaKernel k[8] = {k_mfmamix<1, NS>, k_mfmamix<2, NS>, k_mfmamix<3, NS>, k_mfmamix<4, NS>,
                                  k_mfmamix<5, NS>, k_mfmamix<6, NS>, k_mfmamix<7, NS>, k_mfmamix<8, NS>};
  return k[nr - 1];
}

constexpr int kParts = 3;
constexpr int kPerCU = 2;

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
  const int grid = std::min(cus * kPerCU, p.ntiles);
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

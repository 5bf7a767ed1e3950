// Gather-mix of the routed experts (Eq. 5) and the residual output (Eq. 6)
// for NCHW bfloat16 inputs with C <= 256, given the coefficients alpha.
//
// Tiles.  Image b is cut into nt = ceil(HW / 64) tiles of 64 positions by all
// C channels.  A 512-thread workgroup holds one tile in LDS, widened to
// float32, and every routed expert reads its k support rows from there: the
// gather costs one 16-byte LDS read per support entry and lane (4 positions),
// so each loaded channel row serves every expert whose support contains it.
// Two workgroups share a CU (about 77 KB of LDS each).
//
// Schedule.  Workgroup g of G takes the contiguous run of tiles
// [g * ntiles / G, (g + 1) * ntiles / G), which mostly lies in one image, so
// the image's coefficients are loaded into LDS only when the image changes
// (one step ahead, in registers).  While tile n is mixed, the data of tile
// n + 1 is already in registers and the loads of tile n + 2 are in flight.
//
// Waits.  Loads and stores share one in-order counter.  The experts of a tile
// are computed in a fixed number of passes whose results stay in registers
// until the next tile has been written to LDS, and only then are they
// stored, so that the compiler's wait for the next tile's data counts exactly
// the operations issued after it and never drains the loads still in flight.
//
// Mixing.  Each quarter wave computes one expert (or the residual) for the 64
// positions of the tile, each lane 4 consecutive positions.  The byte offsets
// of an expert's support rows are 16-bit values in LDS read four at a time,
// and so are the coefficients.
#include <algorithm>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kTT = 64;             // positions per tile
constexpr int kRowBytes = kTT * 4;  // bytes of one channel row of the LDS tile
constexpr int kPerCU = 2;           // workgroups per CU
constexpr int kMaxLds = 80 * 1024 - 1024;
constexpr int kASlots = 4;          // coefficients per thread prefetched in registers
constexpr int kExpertsPerPass = 4 * kWaves;

struct TileArgs {
  int B, C, HW, E, R, k, kq, nU;  // kq: k rounded up to a multiple of 4
  int nt, ntiles;                 // tiles per image, tiles in the batch
};

// LDS regions in bytes: tile [C][kTT] float, coefficients [R][kq] float,
// support row offsets [R][kq] uint16.
struct TileLds {
  size_t alpha, sofs, total;
};

__host__ __device__ inline TileLds tile_lds(int C, int R, int kq) {
  TileLds l;
  l.alpha = (size_t)C * kTT * 4;
  l.sofs = l.alpha + (size_t)R * kq * 4;
  l.total = l.sofs + (((size_t)R * kq * 2 + 15) & ~(size_t)15);
  return l;
}

// Issues the global loads of tile n into buf (4 x 16 bytes per thread): thread
// t reads 8 positions of channel (t >> 3) + 64u in round u.  Every round
// loads (rows past C repeat row C - 1, positions past the image repeat its
// last vector), so the loads are straight-line code; the surplus is never
// written to an output.
__device__ __forceinline__ void issue_tile(const TileArgs& p, const uint16_t* __restrict__ x, int n, uint4* buf) {
  const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
  const int p0 = j * kTT;
  const int vvalid = min(kTT, p.HW - p0) / 8;
  const uint16_t* xb = x + (int64_t)b * p.C * p.HW + p0;
  const int qv = threadIdx.x & 7;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = (threadIdx.x >> 3) + u * 64;
    buf[u] = *reinterpret_cast<const uint4*>(xb + (int64_t)min(c, p.C - 1) * p.HW + min(qv, vvalid - 1) * 8);
  }
}

// Widens tile data into the LDS tile (channels < C).
__device__ __forceinline__ void store_tile(const TileArgs& p, const uint4* buf, float* tile) {
  const int qv = threadIdx.x & 7;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = (threadIdx.x >> 3) + u * 64;
    if (u * 64 < p.C && c < p.C) {
      float4* dst = reinterpret_cast<float4*>(tile + c * kTT + qv * 8);
      dst[0] = make_float4(bf16_lo(buf[u].x), bf16_hi(buf[u].x), bf16_lo(buf[u].y), bf16_hi(buf[u].y));
      dst[1] = make_float4(bf16_lo(buf[u].z), bf16_hi(buf[u].z), bf16_lo(buf[u].w), bf16_hi(buf[u].w));
    }
  }
}

// Coefficient e of image b in the padded [R][kq] layout (0 for padding),
// read from alpha [B][R][k].
__device__ __forceinline__ float alpha_entry(const TileArgs& p, const float* __restrict__ alpha, int b, int e) {
  const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
  const int64_t rk = (int64_t)p.R * p.k;
  const float v = alpha[min((int64_t)b * rk + (int64_t)o * p.k + i, (int64_t)p.B * rk - 1)];
  return (o < p.R && i < p.k) ? v : 0.f;
}

// y[o][p0 + 4 l .. +3] of one routed expert from lane l of a quarter wave: K
// (or kq, when K == 0) support entries, each a 16-byte read of the LDS tile at
// the entry's 16-bit byte offset plus the lane's own.  Padding entries have
// coefficient 0 and row 0.
template <int K>
__device__ __forceinline__ float4 mix_expert(const uint16_t* ofs, const float* al, const char* base, int kq) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  const int n = K > 0 ? K : kq;
  // the offsets and coefficients of the next four entries are read while the
  // rows of the current four are in flight (the last step reads its own again)
  uint2 of = *reinterpret_cast<const uint2*>(ofs);
  float4 a = *reinterpret_cast<const float4*>(al);
  auto step4 = [&](int i) {
    const int inext = min(i + 4, n - 4);
    const uint2 of_n = *reinterpret_cast<const uint2*>(ofs + inext);
    const float4 a_n = *reinterpret_cast<const float4*>(al + inext);
    // keep the two reads above ahead of the row reads below
    __builtin_amdgcn_sched_barrier(0);
    const float4 v0 = *reinterpret_cast<const float4*>(base + (of.x & 0xffffu));
    const float4 v1 = *reinterpret_cast<const float4*>(base + (of.x >> 16));
    const float4 v2 = *reinterpret_cast<const float4*>(base + (of.y & 0xffffu));
    const float4 v3 = *reinterpret_cast<const float4*>(base + (of.y >> 16));
#define MOCE_FMA4(A, V) \
    acc.x = fmaf(A, V.x, acc.x); acc.y = fmaf(A, V.y, acc.y); acc.z = fmaf(A, V.z, acc.z); acc.w = fmaf(A, V.w, acc.w)
    MOCE_FMA4(a.x, v0); MOCE_FMA4(a.y, v1); MOCE_FMA4(a.z, v2); MOCE_FMA4(a.w, v3);
#undef MOCE_FMA4
    of = of_n;
    a = a_n;
  };
  if constexpr (K > 0) {
#pragma unroll 2
    for (int i = 0; i < K; i += 4) step4(i);
  } else {
    for (int i = 0; i < n; i += 4) step4(i);
  }
  return acc;
}

// The residual output for lane l of a quarter wave: mean of the tile rows of
// the uncovered channels U, exactly 0 when U is empty.
__device__ __forceinline__ float4 residual(const int32_t* __restrict__ U, int nU, const char* base) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int u = 0; u < nU; ++u) {
    const float4 v = *reinterpret_cast<const float4*>(base + U[u] * kRowBytes);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  if (nU > 0) {
    const float n = (float)nU;
    acc = make_float4(acc.x / n, acc.y / n, acc.z / n, acc.w / n);
  }
  return acc;
}

__device__ __forceinline__ uint2 pack_bf16x4(float4 v) {
  return make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
}

// K: kq when fixed (else 0); NP: passes of kExpertsPerPass experts covering
// the R routed experts and the residual (else 0: a runtime loop).
template <int K, int NP>
__global__ void __launch_bounds__(kThreads, 2 * kPerCU)
k_tilemix(TileArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, const int32_t* __restrict__ s,
          const float* __restrict__ alpha, const int32_t* __restrict__ U) {
  extern __shared__ __align__(16) unsigned char smem[];
  const TileLds ll = tile_lds(p.C, p.R, p.kq);
  float* tile = reinterpret_cast<float*>(smem);                  // [C][kTT]
  float* al = reinterpret_cast<float*>(smem + ll.alpha);         // [R][kq]
  uint16_t* sofs = reinterpret_cast<uint16_t*>(smem + ll.sofs);  // [R][kq]

  const int G = gridDim.x;
  const int t0 = (int)((int64_t)blockIdx.x * p.ntiles / G);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * p.ntiles / G);
  if (t0 >= t1) return;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rkq = p.R * p.kq;

  // The first two tiles' loads go out first; the support offsets and the
  // first image's coefficients are then read with all loads issued before
  // any is used, so the prologue costs about one memory round trip.
  uint4 bufa[4], bufb[4];
  issue_tile(p, x, t0, bufa);
  if (t0 + 1 < t1) issue_tile(p, x, t0 + 1, bufb);
  int cur = t0 / p.nt;
  const bool pre = rkq <= kASlots * kThreads;  // a full table fits kASlots values per thread
  if (pre) {
    int32_t sv[kASlots];
    float av[kASlots];
#pragma unroll
    for (int q = 0; q < kASlots; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      sv[q] = s[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)];
      av[q] = alpha[min((int64_t)cur * p.R * p.k + (int64_t)o * p.k + i, (int64_t)p.B * p.R * p.k - 1)];
    }
#pragma unroll
    for (int q = 0; q < kASlots; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      if (e < rkq) {
        const bool valid = o < p.R && i < p.k;
        sofs[e] = (uint16_t)((valid ? sv[q] : 0) * kRowBytes);
        al[e] = valid ? av[q] : 0.f;
      }
    }
  } else {
    for (int e = threadIdx.x; e < rkq; e += kThreads) {
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      const int32_t sv = s[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)];
      sofs[e] = (uint16_t)((i < p.k ? sv : 0) * kRowBytes);
      al[e] = alpha_entry(p, alpha, cur, e);
    }
  }
  store_tile(p, bufa, tile);
  __syncthreads();

  float an[kASlots];
  const int gq = lane >> 4, l4 = lane & 15;
  const char* base = reinterpret_cast<const char*>(tile) + l4 * 16;

  // One step with tile n in LDS and the data of tile n + 1 (if any) in nxt:
  // fetch the next image's coefficients if it starts at n + 1, start the
  // loads of n + 2 into spare, mix n, move n + 1 into LDS, store n's outputs.
  auto step = [&](int n, uint4* nxt, uint4* spare) {
    const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
    const int n1 = n + 1, n2 = n + 2;
    if (b != cur) {
      // the image changed at this tile: its coefficients were fetched in the
      // previous step (or are read now when they do not fit the registers)
      if (pre) {
#pragma unroll
        for (int q = 0; q < kASlots; ++q) {
          const int e = threadIdx.x + q * kThreads;
          if (e < rkq) al[e] = an[q];
        }
      } else {
        for (int e = threadIdx.x; e < rkq; e += kThreads) al[e] = alpha_entry(p, alpha, b, e);
      }
      cur = b;
      __syncthreads();
    }
    const int b1 = n1 / p.nt;
    if (pre && n1 < t1 && b1 != b) {
#pragma unroll
      for (int q = 0; q < kASlots; ++q) an[q] = alpha_entry(p, alpha, b1, threadIdx.x + q * kThreads);
    }
    if (n2 < t1) issue_tile(p, x, n2, spare);

    const int p0 = j * kTT;
    const bool store = l4 * 4 < min(kTT, p.HW - p0);  // H*W is a multiple of 8: all four positions or none
    uint16_t* yb = y + (int64_t)b * p.E * p.HW + p0 + l4 * 4;
    constexpr int NPC = NP > 0 ? NP : 1;
    float4 res[NPC];
    const int np = NP > 0 ? NP : (p.R + 1 + kExpertsPerPass - 1) / kExpertsPerPass;
    // with NP fixed, every pass's result is kept and stored after the tile
    // move; with a runtime pass count, each pass stores its own result
#pragma unroll
    for (int q = 0; q < NPC; ++q) {
      for (int qq = (NP > 0 ? q : 0); qq < (NP > 0 ? q + 1 : np); ++qq) {
        const int o = 4 * wv + qq * kExpertsPerPass + gq;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        if (o < p.R)
          acc = mix_expert<K>(sofs + o * p.kq, al + o * p.kq, base, p.kq);
        else if (o == p.R)
          acc = residual(U, p.nU, base);
        if (NP > 0)
          res[q] = acc;
        else if (store && o <= p.R)
          *reinterpret_cast<uint2*>(yb + (int64_t)o * p.HW) = pack_bf16x4(acc);
      }
    }
    __syncthreads();  // every wave is done with the LDS tile
    if (n1 < t1) store_tile(p, nxt, tile);
    if (NP > 0) {
#pragma unroll
      for (int q = 0; q < NPC; ++q) {
        const int o = 4 * wv + q * kExpertsPerPass + gq;
        if (store && o <= p.R) *reinterpret_cast<uint2*>(yb + (int64_t)o * p.HW) = pack_bf16x4(res[q]);
      }
    }
    __syncthreads();
  };

  // two steps per trip, so that the two register buffers trade roles
  // without being copied
  for (int n = t0;;) {
    step(n, bufb, bufa);
    if (++n >= t1) break;
    step(n, bufa, bufb);
    if (++n >= t1) break;
  }
}

int rounded_k(const Shape& sh) { return (sh.k + 3) & ~3; }

int64_t tiles_per_image(const Shape& sh) { return (sh.HW + kTT - 1) / kTT; }

using TileKernel = void (*)(TileArgs, const uint16_t*, uint16_t*, const int32_t*, const float*, const int32_t*);

TileKernel pick_kernel(const Shape& sh) {
  const int kq = rounded_k(sh);
  const int np = (sh.R + 1 + kExpertsPerPass - 1) / kExpertsPerPass;
  if (kq == 32 && np == 1) return k_tilemix<32, 1>;
  if (kq == 32 && np == 2) return k_tilemix<32, 2>;
  if (kq == 64 && np == 2) return k_tilemix<64, 2>;
  return k_tilemix<0, 0>;
}

}  // namespace

size_t tilemix_lds_bytes(const Shape& sh) { return tile_lds((int)sh.C, sh.R, rounded_k(sh)).total; }

bool tilemix_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.HW % 8 != 0 || sh.C > 256) return false;
  if (sh.B * tiles_per_image(sh) > INT32_MAX / 2) return false;
  return tilemix_lds_bytes(sh) <= (size_t)kMaxLds;
}

hipError_t launch_tilemix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st) {
  TileArgs p;
  p.B = (int)sh.B;
  p.C = (int)sh.C;
  p.HW = (int)sh.HW;
  p.E = sh.E;
  p.R = sh.R;
  p.k = sh.k;
  p.kq = rounded_k(sh);
  p.nU = nU;
  p.nt = (int)tiles_per_image(sh);
  p.ntiles = (int)(sh.B * p.nt);

  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  const int grid = (int)std::min<int64_t>((int64_t)cus * kPerCU, p.ntiles);
  const size_t lds = tilemix_lds_bytes(sh);
  const TileKernel kern = pick_kernel(sh);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, st, p, static_cast<const uint16_t*>(x),
                     static_cast<uint16_t*>(y), s, alpha, U);
  return hipGetLastError();
}

}  // namespace moce

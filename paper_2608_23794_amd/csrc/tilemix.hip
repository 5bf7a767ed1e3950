// Gather-mix of the routed experts (Eq. 5) and the residual output (Eq. 6)
// for NCHW bfloat16 inputs with C <= 256, given the coefficients alpha.
//
// The tile and the expert mix are those of tile_common.h; two workgroups share
// a CU (about 77 KB of LDS each).
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
#include <algorithm>

#include "tile_common.h"

namespace moce {
namespace {

using namespace tile;

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
  const bool dyn = p.nUb != nullptr;
  // the support rows of image b (the same rows for every image when static)
  auto srows = [&](int b) { return dyn ? s + (int64_t)b * p.R * p.k : s; };

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
    const int32_t* sr = srows(cur);
#pragma unroll
    for (int q = 0; q < kASlots; ++q) {
      const int e = threadIdx.x + q * kThreads;
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      sv[q] = min(max(sr[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)], 0), p.C - 1);
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
    const int32_t* sr = srows(cur);
    for (int e = threadIdx.x; e < rkq; e += kThreads) {
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      const int32_t sv = min(max(sr[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)], 0), p.C - 1);
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
      if (dyn) {  // the image's own supports
        const int32_t* sr = srows(b);
        for (int e = threadIdx.x; e < rkq; e += kThreads) {
          const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
          const int32_t sv = min(max(sr[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)], 0), p.C - 1);
          sofs[e] = (uint16_t)((o < p.R && i < p.k ? sv : 0) * kRowBytes);
        }
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
          acc = dyn ? residual(U + (int64_t)b * p.C, p.nUb[b], base) : residual(U, p.nU, base);
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

// Register-resident variant (tile_common.h) for k <= 16 NR and
// R + 1 <= NP * kExpertsPerPass: the lanes hold the coefficients and support
// row offsets, and LDS holds only the tile.  Same schedule as k_tilemix; the
// next image's coefficients are prefetched into registers one step ahead,
// and padding entries are zeroed where the values are used, not right after
// the loads.
template <int NR, int NP>
__global__ void __launch_bounds__(kThreads, 2 * kPerCU)
k_tilemix_regs(TileArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, const int32_t* __restrict__ s,
               const float* __restrict__ alpha, const int32_t* __restrict__ U) {
  extern __shared__ __align__(16) unsigned char smem[];
  float* tile = reinterpret_cast<float*>(smem);  // [C][kTT]

  const int G = gridDim.x;
  const int t0 = (int)((int64_t)blockIdx.x * p.ntiles / G);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * p.ntiles / G);
  if (t0 >= t1) return;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int gq = lane >> 4, l4 = lane & 15;

  uint4 bufa[4], bufb[4];
  issue_tile(p, x, t0, bufa);
  if (t0 + 1 < t1) issue_tile(p, x, t0 + 1, bufb);

  // entry m of pass q: expert 4 wv + q kExpertsPerPass + gq, support position l4 + 16 m
  int ofs[NP][NR], eoff[NP][NR];
  uint32_t valid = 0;
#pragma unroll
  for (int q = 0; q < NP; ++q)
#pragma unroll
    for (int m = 0; m < NR; ++m) {
      const int o = 4 * wv + q * kExpertsPerPass + gq, i = l4 + kRowLanes * m;
      const bool v = o < p.R && i < p.k;
      valid |= (uint32_t)v << (q * NR + m);
      eoff[q][m] = v ? o * p.k + i : 0;
      ofs[q][m] = s[eoff[q][m]];
    }
  float a[NP][NR], an[NP][NR];
  auto load_alpha = [&](int b, float (&dst)[NP][NR]) {
    const float* ab = alpha + (int64_t)b * p.R * p.k;
#pragma unroll
    for (int q = 0; q < NP; ++q)
#pragma unroll
      for (int m = 0; m < NR; ++m) dst[q][m] = ab[eoff[q][m]];
  };
  auto take_alpha = [&]() {
#pragma unroll
    for (int q = 0; q < NP; ++q)
#pragma unroll
      for (int m = 0; m < NR; ++m) a[q][m] = (valid >> (q * NR + m)) & 1 ? an[q][m] : 0.f;
  };
  int cur = t0 / p.nt;
  load_alpha(cur, an);
#pragma unroll
  for (int q = 0; q < NP; ++q)
#pragma unroll
    for (int m = 0; m < NR; ++m) ofs[q][m] = (valid >> (q * NR + m)) & 1 ? ofs[q][m] * kRowBytes : 0;
  take_alpha();
  store_tile(p, bufa, tile);
  __syncthreads();
  const char* base = reinterpret_cast<const char*>(tile) + l4 * 16;

  auto step = [&](int n, uint4* nxt, uint4* spare) {
    const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
    const int n1 = n + 1, n2 = n + 2;
    if (b != cur) {
      take_alpha();
      cur = b;
    }
    if (n1 < t1 && n1 / p.nt != b) load_alpha(n1 / p.nt, an);
    if (n2 < t1) issue_tile(p, x, n2, spare);

    const int p0 = j * kTT;
    const bool store = l4 * 4 < min(kTT, p.HW - p0);  // H*W is a multiple of 8: all four positions or none
    uint16_t* yb = y + (int64_t)b * p.E * p.HW + p0 + l4 * 4;
    float4 res[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int o = 4 * wv + q * kExpertsPerPass + gq;
      res[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (o < p.R)
        res[q] = mix_expert_regs<NR>(a[q], ofs[q], base);
      else if (o == p.R)
        res[q] = residual(U, p.nU, base);
    }
    __syncthreads();  // every wave is done with the LDS tile
    if (n1 < t1) store_tile(p, nxt, tile);
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int o = 4 * wv + q * kExpertsPerPass + gq;
      if (store && o <= p.R) *reinterpret_cast<uint2*>(yb + (int64_t)o * p.HW) = pack_bf16x4(res[q]);
    }
    __syncthreads();
  };

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

int expert_passes(const Shape& sh) { return (sh.R + 1 + kExpertsPerPass - 1) / kExpertsPerPass; }

// register rows per expert for the register-resident kernel, 0 when it does not apply
int regs_rows(const Shape& sh) {
  if (sh.k > 4 * kRowLanes || expert_passes(sh) > 2) return 0;
  return (sh.k + kRowLanes - 1) / kRowLanes;
}

TileKernel pick_kernel(const Shape& sh) {
  const int nr = regs_rows(sh), np = expert_passes(sh);
  if (nr > 0) {
    static const TileKernel regs[4][2] = {{k_tilemix_regs<1, 1>, k_tilemix_regs<1, 2>},
                                          {k_tilemix_regs<2, 1>, k_tilemix_regs<2, 2>},
                                          {k_tilemix_regs<3, 1>, k_tilemix_regs<3, 2>},
                                          {k_tilemix_regs<4, 1>, k_tilemix_regs<4, 2>}};
    return regs[nr - 1][np - 1];
  }
  // k <= 64 with at most two expert passes always takes the register
  // kernel above, so only the general form is instantiated here
  return k_tilemix<0, 0>;
}

}  // namespace

size_t tilemix_lds_bytes(const Shape& sh) {
  if (regs_rows(sh) > 0) return (size_t)sh.C * kRowBytes;
  return tile_lds((int)sh.C, sh.R, rounded_k(sh)).total;
}

bool tilemix_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.HW % 8 != 0 || sh.C > 256) return false;
  if (sh.B * tiles_per_image(sh) > INT32_MAX / 2) return false;
  return tilemix_lds_bytes(sh) <= (size_t)kMaxLds;
}

namespace {

hipError_t tilemix_launch(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, const int32_t* nUb, void* y, hipStream_t st) {
  TileArgs p;
  p.nUb = nUb;
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
  // input-conditioned supports take the LDS-table kernel, which reloads the
  // support rows when the image changes
  const size_t lds = nUb ? tile_lds((int)sh.C, sh.R, rounded_k(sh)).total : tilemix_lds_bytes(sh);
  const TileKernel kern = nUb ? k_tilemix<0, 0> : pick_kernel(sh);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, st, p, static_cast<const uint16_t*>(x),
                     static_cast<uint16_t*>(y), s, alpha, U);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tilemix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st) {
  return tilemix_launch(sh, x, s, alpha, U, nU, nullptr, y, st);
}

bool tilemix_dynamic_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.HW % 8 != 0 || sh.C > 256) return false;
  if (sh.B * tiles_per_image(sh) > INT32_MAX / 2) return false;
  return tile_lds((int)sh.C, sh.R, rounded_k(sh)).total <= (size_t)kMaxLds;
}

hipError_t launch_tilemix_dynamic(const Shape& sh, const void* x, const int32_t* S, const float* alpha,
                                  const int32_t* U, const int32_t* nU, void* y, hipStream_t st) {
  return tilemix_launch(sh, x, S, alpha, U, 0, nU, y, st);
}

}  // namespace moce

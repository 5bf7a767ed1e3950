// Device pieces of the tile kernels (tilemix.hip): the LDS
// tile of 64 positions by all C channels held as float32, its loads and
// stores, and the quarter-wave expert mix that reads it.
//
// Tiles.  Image b is cut into nt = ceil(HW / 64) tiles of 64 positions by all
// C channels.  A 512-thread workgroup holds one tile in LDS, widened to
// float32, and every routed expert reads its k support rows from there: the
// gather costs one 16-byte LDS read per support entry and lane (4 positions),
// so each loaded channel row serves every expert whose support contains it.
//
// Mixing.  Each quarter wave computes one expert (or the residual) for the 64
// positions of the tile, each lane 4 consecutive positions.  The byte offsets
// of an expert's support rows are 16-bit values in LDS read four at a time,
// and so are the coefficients.
#pragma once

#include "moce_internal.h"

namespace moce {
namespace tile {

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
  // input-conditioned supports: per image rows s[b][R][k], uncovered lists
  // U[b][C] and counts nUb[b] (null for the static supports)
  const int32_t* nUb;
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

// Issues the global loads of tile n into buf (2048 / NTH x 16 bytes per
// thread for a workgroup of NTH threads): thread t reads 8 positions of
// channel (t >> 3) + (NTH / 8) u in round u.  Every round loads (rows past C
// repeat row C - 1, positions past the image repeat its last vector), so the
// loads are straight-line code; the surplus is never written to an output.
template <int NTH = kThreads>
__device__ __forceinline__ void issue_tile(const TileArgs& p, const uint16_t* __restrict__ x, int b, int j,
                                           uint4* buf, int tid = threadIdx.x) {
  constexpr int kRounds = 256 * 8 / NTH;
  const int p0 = j * kTT;
  const int vvalid = min(kTT, p.HW - p0) / 8;
  const uint16_t* xb = x + (int64_t)b * p.C * p.HW + p0;
  const int qv = tid & 7;
#pragma unroll
  for (int u = 0; u < kRounds; ++u) {
    const int c = (tid >> 3) + u * (NTH / 8);
    buf[u] = *reinterpret_cast<const uint4*>(xb + (int64_t)min(c, p.C - 1) * p.HW + min(qv, vvalid - 1) * 8);
  }
}

// The same for tile n = b * nt + j.
template <int NTH = kThreads>
__device__ __forceinline__ void issue_tile(const TileArgs& p, const uint16_t* __restrict__ x, int n, uint4* buf,
                                           int tid = threadIdx.x) {
  issue_tile<NTH>(p, x, n / p.nt, n - (n / p.nt) * p.nt, buf, tid);
}

// Widens tile data into the LDS tile (channels < C).
template <int NTH = kThreads>
__device__ __forceinline__ void store_tile(const TileArgs& p, const uint4* buf, float* tile) {
  constexpr int kRounds = 256 * 8 / NTH;
  const int qv = threadIdx.x & 7;
#pragma unroll
  for (int u = 0; u < kRounds; ++u) {
    const int c = (threadIdx.x >> 3) + u * (NTH / 8);
    if (u * (NTH / 8) < p.C && c < p.C) {
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

// Register-resident experts.  The 16 lanes of a quarter wave form one DPP
// row; for the expert it computes, lane l holds the coefficients and support
// row byte offsets of entries l, l + 16, ..., l + 16 (NR - 1) (coefficient 0
// and row 0 past k).  Entry i is broadcast from lane i % 16 of the row with
// row_newbcast, which the compiler folds into the LDS address add, so LDS
// carries only the tile rows: 16 bytes per lane for four FMAs.
constexpr int kRowLanes = 16;

template <int I>
__device__ __forceinline__ int row_bcast(int v) {
  return __builtin_amdgcn_mov_dpp(v, 0x150 + I, 0xf, 0xf, true);
}
template <int I>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(row_bcast<I>(__float_as_int(v)));
}

// Rows of the four entries 4 G .. 4 G + 3 (G counts groups of four over all
// NR registers).
template <int G>
__device__ __forceinline__ void read_group(float4 (&v)[4], const int* ofs, const char* base) {
  constexpr int m = G / 4, i = 4 * (G % 4);
  v[0] = *reinterpret_cast<const float4*>(base + row_bcast<i>(ofs[m]));
  v[1] = *reinterpret_cast<const float4*>(base + row_bcast<i + 1>(ofs[m]));
  v[2] = *reinterpret_cast<const float4*>(base + row_bcast<i + 2>(ofs[m]));
  v[3] = *reinterpret_cast<const float4*>(base + row_bcast<i + 3>(ofs[m]));
}

template <int G>
__device__ __forceinline__ void fma_group(float4& acc, const float4 (&v)[4], const float* a) {
  constexpr int m = G / 4, i = 4 * (G % 4);
  const float A[4] = {row_bcast<i>(a[m]), row_bcast<i + 1>(a[m]), row_bcast<i + 2>(a[m]), row_bcast<i + 3>(a[m])};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    acc.x = fmaf(A[u], v[u].x, acc.x);
    acc.y = fmaf(A[u], v[u].y, acc.y);
    acc.z = fmaf(A[u], v[u].z, acc.z);
    acc.w = fmaf(A[u], v[u].w, acc.w);
  }
}

// Groups G .. 4 NR - 1, the rows of group G already read into cur: the next
// group's rows are read before this group's FMAs (the scheduling barrier
// keeps that order).
template <int G, int NR>
__device__ __forceinline__ void mix_groups(float4& acc, const float* a, const int* ofs, const char* base,
                                           const float4 (&cur)[4]) {
  if constexpr (G + 1 < 4 * NR) {
    float4 nxt[4];
    read_group<G + 1>(nxt, ofs, base);
    __builtin_amdgcn_sched_barrier(0);
    fma_group<G>(acc, cur, a);
    mix_groups<G + 1, NR>(acc, a, ofs, base, nxt);
  } else {
    fma_group<G>(acc, cur, a);
  }
}

// y[o][p0 + 4 l .. +3] of the routed expert whose entries the row holds.
// Every lane of the row must be active.
template <int NR>
__device__ __forceinline__ float4 mix_expert_regs(const float* a, const int* ofs, const char* base) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 v[4];
  read_group<0>(v, ofs, base);
  mix_groups<0, NR>(acc, a, ofs, base, v);
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

}  // namespace tile
}  // namespace moce

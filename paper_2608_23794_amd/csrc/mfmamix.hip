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
// Work split.  One workgroup per CU walks a contiguous range of tiles (64
// positions x all C channels of one image) with three kinds of waves, so
// that no wave that computes ever waits behind the memory system; each kind
// runs its own loop over the tiles, and all waves meet at one barrier per
// tile.  Two loader waves copy each tile straight into a ring of four LDS
// tile buffers (global-to-LDS loads, no registers; in the forward x mostly
// comes back from the infinity cache, where the pooling kernel left it),
// keeping up to three tiles in flight, and wait for their own copies with
// explicit counters.  Four consumer waves only compute: wave w multiplies
// experts 16 w .. 16 w + 15 at all 64 positions, holding its 16 rows of A_b
// (all channels, every part) in registers as MFMA B operands and reading the
// x tile as MFMA A operands with the transposing LDS read, which turns the
// position-contiguous channel rows into channel-contiguous operands; results
// go to an LDS output buffer.  Two store waves write the previous tile's
// results from there to y, whole 128-byte rows per store.  The tile copies
// and the stores of y carry the non-temporal hint.  At the first tile each
// consumer wave builds its rows of A_b through the last ring buffer, still
// free then; when the image changes it rebuilds them, 8 at a time, in its own
// staging area, while the other waves carry on.
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

constexpr int kConsumers = 4;                   // waves computing products
constexpr int kLoaders = 2;                     // waves copying tiles into LDS
constexpr int kStorers = 2;                     // waves writing results to y
constexpr int kCThreads = 64 * kConsumers;
constexpr int kLThreads = 64 * kLoaders;
constexpr int kThreads = 64 * (kConsumers + kLoaders + kStorers);
constexpr int kRing = 4;                        // LDS tile buffers
constexpr int kTile = 64;                       // positions per tile
constexpr int kRow = kTile * 2;                 // bytes of one channel row of an LDS tile
constexpr int kMaxE = 64;                       // rows of A_b
constexpr int kStageRows = 8;                   // rows of A_b a consumer wave assembles at a time
constexpr int kMaxC = 256;
constexpr int kPre = 8;                         // coefficient entries per consumer lane fetched ahead
constexpr int kUPer = kMaxC / 64;               // uncovered channels per lane of the residual's wave
constexpr int kExpertsPerWave = 16;
static_assert(kExpertsPerWave == 2 * kStageRows, "a rebuild takes two groups of staging rows");
constexpr int kOutWave = kExpertsPerWave * kRow;  // one consumer wave's results for a tile

// Workgroup barrier for LDS traffic: waits for this wave's own LDS (and
// scalar) accesses, then for every wave.  Unlike __syncthreads it does not
// wait for outstanding global-to-LDS copies (the release fence would drain
// the whole ring of tiles in flight at every step); each copy is waited for
// explicitly, with vm_wait, before the barrier that publishes its tile.  The
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// s_waitcnt operand that waits until at most n vector memory accesses of
// this wave are outstanding (the LDS/scalar and export counters left at
// their maxima)
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Cache-policy operand of the global-to-LDS load: the non-temporal bit.
constexpr int kCachePolicyNT = 2;

struct MixArgs {
  int C, HW, E, R, k, nU, nt, ntiles;
  Epi ep;   // output epilogue, applied to the accumulators before rounding
};

// LDS: the ring of x tiles [C][kTile] bf16, each consumer wave's A_b staging
// rows [kStageRows][C] bf16, then two output buffers [E rows][kTile] bf16
// (the consumer waves' results of alternate tiles; 16-byte chunk q of row r
// is stored at chunk q ^ (r & 7)).
__host__ __device__ inline size_t mfma_lds(int C) {
  return (size_t)kRing * C * kRow + (size_t)kConsumers * kStageRows * C * 2 + (size_t)2 * kConsumers * kOutWave;
}

// Chunk q (16 bytes = 8 positions) of channel row c of a tile is stored at
// chunk q ^ tile_swz(c).  One transposing read fetches 8 bytes per lane from
// rows 8 g + 4 h + (l >> 2) (+ 32 ks) of 16-lane group g, two chunks per row;
// with 64 banks of 4 bytes, rows of equal parity collide unless their chunks
// differ, so the swizzle takes bits 1 and 3 of the row: the 16 lanes of a
// group, and the 32 of two neighbouring groups, then fall on distinct banks.
__device__ __forceinline__ int tile_swz(int c) { return (((c >> 1) & 1) << 1) | (((c >> 3) & 1) << 2); }

// Byte offset of A_b[o][c] in a staging area [rows][C] bf16 (C = 32 NR),
// whose 16-byte chunks are rotated by 4 (o & 3) within the row so that the
// operand reads (16 rows x 64 bytes) spread over the banks.  C is a constant
// of the kernel, so the row size and the rotation's wrap (c / 8 < C / 8 and
// 4 (o & 3) <= 12) cost a few full-rate operations.
template <int NR>
__device__ __forceinline__ int stage_off(int o, int c) {
  constexpr int nch = 4 * NR;  // 16-byte chunks per row
  int ch = (c >> 3) + 4 * (o & 3);
  if constexpr ((nch & (nch - 1)) == 0) {
    ch &= nch - 1;
  } else {
#pragma unroll
    for (int t = 0; t <= 11 / nch; ++t) ch = ch >= nch ? ch - nch : ch;
  }
  return o * (64 * NR) + ch * 16 + (c & 7) * 2;
}

// Copies tile n into the LDS tile buffer `buf` with global-to-LDS loads, one
// 16-byte load per loader lane and round: loader lane t (of 128) fills slot t
// of each 2 KB block u, i.e. chunk t & 7 of row (t >> 3) + 16 u, with the 8
// positions of the tile that belong there under the swizzle.  Positions past
// the image repeat its last vector; those outputs are never stored.  This is
// the last read of x in the forward, so the loads carry the non-temporal hint
// (together with the non-temporal stores below the forward at the ResNet-50
// stage-1 shape runs 3.5 us faster; the pool kernel reads x normally, so the
// image it pooled is in the infinity cache for these reads).
template <int NR>
__device__ __forceinline__ void copy_tile(const MixArgs& p, const uint16_t* __restrict__ x, int n, unsigned char* buf,
                                          int lt) {
  const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
  const int p0 = j * kTile;
  const int qmax = min(kTile, p.HW - p0) / 8 - 1;
  const uint16_t* src = x + ((int64_t)b * p.C + (lt >> 3)) * p.HW + p0;
  MOCE_LDS unsigned char* dst = (MOCE_LDS unsigned char*)buf + (lt & ~63) * 16;
#pragma unroll
  for (int u = 0; u < 2 * NR; ++u) {
    const int q = min((lt & 7) ^ tile_swz((lt >> 3) + 16 * u), qmax);
    __builtin_amdgcn_global_load_lds((const void*)(src + (int64_t)u * 16 * p.HW + q * 8),
                                     (MOCE_LDS void*)(dst + u * 16 * kRow), 16, 0, kCachePolicyNT);
  }
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

// A consumer wave's coefficients.  Entry i < 16 k of wave w is coefficient
// i % k of expert 16 w + i / k, i.e. entry 16 w k + i of an image's flattened
// [R][k] block; lane l handles entries l + 64 r.  slot[] holds their staging
// slots, 16 bits each: the byte offset of the entry in a staging area of the
// wave's 16 rows (below 32 C <= 8192), 0xffff for none.  uslot[] does the
// same for the residual row's uncovered channels l + 64 u (only in the wave
// holding row R).
struct WaveCoefs {
  float a[kPre];
  uint32_t slot[kPre / 2];
  uint32_t uslot[kUPer / 2];
};

__device__ __forceinline__ uint32_t half_of(uint32_t packed, int r) { return (packed >> (16 * (r & 1))) & 0xffffu; }

// A lane's share of the wave's support indices (entries l + 64 r) and of the
// uncovered channels (l + 64 u; U may be null when nU == 0, and s is read
// instead).  The caller pins the results with empty asm statements, so that
// every load is unconditional and all are issued before any is used: left to
// itself the compiler moves each load into the branch that uses it and waits
// for it there, one memory round trip per load.
__device__ __forceinline__ void load_indices(const MixArgs& p, const int32_t* __restrict__ s,
                                             const int32_t* __restrict__ U, int (&cs)[kPre], int (&cu)[kUPer], int cw,
                                             int lane) {
  const int nent = p.R * p.k;
#pragma unroll
  for (int r = 0; r < kPre; ++r) cs[r] = s[min(kExpertsPerWave * cw * p.k + lane + 64 * r, nent - 1)];
#pragma unroll
  for (int u = 0; u < kUPer; ++u) cu[u] = *(p.nU > 0 ? U + min(lane + 64 * u, p.nU - 1) : s);
}

template <int NR>
__device__ __forceinline__ void wave_slots(const MixArgs& p, const int (&cs)[kPre], const int (&cu)[kUPer],
                                           WaveCoefs& wc, int cw, int lane) {
  const int nent = p.R * p.k;
  const float rk = 1.f / (float)p.k;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const int i = lane + 64 * r;
    const int e = kExpertsPerWave * cw * p.k + i;
    // i / k where it is used (i < 16 k): the float quotient of i + 1/2 is
    // below 16 with a relative error of a few ulp, far inside its distance
    // of at least 1 / (2 k) from an integer
    const int eo = (int)(((float)i + 0.5f) * rk);
    // computed for every lane and then selected: branch-free, so that this
    // arithmetic can interleave with other work
    int off = stage_off<NR>(eo & (kExpertsPerWave - 1), cs[r]);
    asm volatile("" : "+v"(off));
    const uint32_t v = (i < kExpertsPerWave * p.k && e < nent) ? (uint32_t)off : 0xffffu;
    wc.slot[r >> 1] = (r & 1) ? (wc.slot[r >> 1] | v << 16) : v;
  }
  const int ro = p.R - kExpertsPerWave * cw;  // the residual row within this wave's experts
#pragma unroll
  for (int u = 0; u < kUPer; ++u) {
    int off = stage_off<NR>(ro & (kExpertsPerWave - 1), cu[u]);
    asm volatile("" : "+v"(off));
    const uint32_t v = (ro >= 0 && ro < kExpertsPerWave && lane + 64 * u < p.nU) ? (uint32_t)off : 0xffffu;
    wc.uslot[u >> 1] = (u & 1) ? (wc.uslot[u >> 1] | v << 16) : v;
  }
}

__device__ __forceinline__ void fetch_coefs(const MixArgs& p, const float* __restrict__ alpha, int b, WaveCoefs& wc,
                                            int cw, int lane) {
  const int nent = p.R * p.k;
  const int first = kExpertsPerWave * cw * p.k;
  const float* ab = alpha + (int64_t)b * nent;
#pragma unroll
  for (int r = 0; r < kPre; ++r) wc.a[r] = ab[min(first + lane + 64 * r, nent - 1)];
}

// The softplus-linear gate's inputs, for a forward that evaluates the gate
// inside the mix (Sec. 3.3: temperature from the support's pooled
// descriptors, then the tempered softmax of the logits): pooled descriptors
// d [B][C], prepared logits w [R][k], slopes a [R][k], offsets c [R].
struct GateArgs {
  const float* d;
  const float* w;
  const float* a;
  const float* c;
};

// A lane's share of the gate's parameters (k = 32: round r of lane l is
// coefficient l & 31 of expert 16 w + 2 r + l / 32).
struct WaveGate {
  float av[kPre], wv[kPre], co[kPre];
};

__device__ __forceinline__ void load_gate(const MixArgs& p, const GateArgs& ga, WaveGate& wg, int cw, int lane) {
  const int nent = p.R * p.k;
  const int first = kExpertsPerWave * cw * p.k;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const int e = min(first + lane + 64 * r, nent - 1);
    wg.av[r] = ga.a[e];
    wg.wv[r] = ga.w[e];
    wg.co[r] = ga.c[min(kExpertsPerWave * cw + 2 * r + (lane >> 5), p.R - 1)];
  }
}

// The pooled descriptors at this wave's support entries for image b.
__device__ __forceinline__ void gather_desc(const MixArgs& p, const GateArgs& ga, int b, const int (&cs)[kPre],
                                            float (&dv)[kPre]) {
#pragma unroll
  for (int r = 0; r < kPre; ++r) dv[r] = ga.d[(int64_t)b * p.C + cs[r]];
}

// The value of lane l ^ OFF within 32-lane segments.  Distances 1, 2, 4
// and 8 stay inside a row of 16 lanes and use DPP moves (quad permutations,
// row shifts, a half-row rotation); 16 uses a permute.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}
template <int OFF>
__device__ __forceinline__ float xor_peer(float v, int lane) {
  if constexpr (OFF == 1) {
    return dpp_mov<0xb1>(v);  // quad_perm [1, 0, 3, 2]
  } else if constexpr (OFF == 2) {
    return dpp_mov<0x4e>(v);  // quad_perm [2, 3, 0, 1]
  } else if constexpr (OFF == 4) {
    const float up = dpp_mov<0x104>(v);  // row_shl 4: lane l + 4
    const float dn = dpp_mov<0x114>(v);  // row_shr 4: lane l - 4
    return (lane & 4) ? dn : up;
  } else if constexpr (OFF == 8) {
    return dpp_mov<0x128>(v);  // row_ror 8: lane l ^ 8 within the row
  } else {
    return __shfl_xor(v, OFF, 32);
  }
}

// wave_sum<32> and wave_max<32> of kPre values at once: the same butterfly
// (partners l ^ 16, 8, 4, 2, 1 in that order) for each, with the kPre
// exchanges of a step issued together.
template <int OFF>
__device__ __forceinline__ void seg32_sum_step(float (&v)[kPre], int lane) {
  float o[kPre];
#pragma unroll
  for (int r = 0; r < kPre; ++r) o[r] = xor_peer<OFF>(v[r], lane);
#pragma unroll
  for (int r = 0; r < kPre; ++r) v[r] += o[r];
}
template <int OFF>
__device__ __forceinline__ void seg32_max_step(float (&v)[kPre], int lane) {
  float o[kPre];
#pragma unroll
  for (int r = 0; r < kPre; ++r) o[r] = xor_peer<OFF>(v[r], lane);
#pragma unroll
  for (int r = 0; r < kPre; ++r) v[r] = fmaxf(v[r], o[r]);
}
__device__ __forceinline__ void seg32_sum(float (&v)[kPre], int lane) {
  seg32_sum_step<16>(v, lane);
  seg32_sum_step<8>(v, lane);
  seg32_sum_step<4>(v, lane);
  seg32_sum_step<2>(v, lane);
  seg32_sum_step<1>(v, lane);
}
__device__ __forceinline__ void seg32_max(float (&v)[kPre], int lane) {
  seg32_max_step<16>(v, lane);
  seg32_max_step<8>(v, lane);
  seg32_max_step<4>(v, lane);
  seg32_max_step<2>(v, lane);
  seg32_max_step<1>(v, lane);
}

// The coefficients of this wave's entries: the gate kernel's operations in
// the gate kernel's lane layout (one expert per 32 lanes, coefficient i on
// lane i), so the values are bit-identical to the ones it writes.
__device__ __forceinline__ void wave_gate(const MixArgs& p, const WaveGate& wg, const float (&dv)[kPre],
                                          WaveCoefs& wc, int cw, int lane) {
  const int nent = p.R * p.k;
  const int first = kExpertsPerWave * cw * p.k;
  bool in[kPre];
  float v[kPre], z[kPre];
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    in[r] = first + lane + 64 * r < nent;
    v[r] = in[r] ? wg.av[r] * dv[r] : 0.f;
  }
  seg32_sum(v, lane);
  // the temperatures: the 16 experts' sums gathered on lanes 0..15 (lane
  // 2 r + h holds expert 2 r + h), one softplus for all of them, then each
  // sent back to its expert's 32 lanes
  float gp = 0.f;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const float x = __shfl(v[r] + wg.co[r], (lane & 1) * 32);
    gp = (lane >> 1) == r ? x : gp;
  }
  const float tp = softplusf(gp) + 1e-3f;
  const float rtp = 1.f / tp;
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    z[r] = coef_z(wg.wv[r], __shfl(rtp, 2 * r + (lane >> 5)));
    v[r] = in[r] ? z[r] : -INFINITY;
  }
  seg32_max(v, lane);
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    // evaluated on every lane, then selected (branch-free)
    float ex = coef_e(z[r], v[r]);
    asm volatile("" : "+v"(ex));
    z[r] = in[r] ? ex : 0.f;
    v[r] = z[r];
  }
  seg32_sum(v, lane);
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    float q = coef_alpha(z[r], 1.f / v[r]);
    asm volatile("" : "+v"(q));
    wc.a[r] = in[r] ? q : 0.f;
  }
}

// The exact split a = hi + mid + lo into bf16 parts (with two parts: hi and
// the rounded remainder).
template <int NS>
__device__ __forceinline__ void split_parts(float a, uint16_t (&pt)[NS]) {
  pt[0] = f32_to_bf16(a);
  const float r1 = a - bf16_to_f32(pt[0]);
  pt[1] = f32_to_bf16(r1);
  if constexpr (NS > 2) pt[2] = f32_to_bf16(r1 - bf16_to_f32(pt[1]));
}

// Builds a consumer wave's rows of A_b in registers at the first tile,
// through a staging area of all 16 rows (the last ring buffer, free until
// tile t0 + 3 is requested): zero the rows, then per part scatter part
// `part` of the coefficients (and 1/nU at the uncovered channels) and read
// the MFMA B operands.  Every part lands on the same slots, so one zeroing
// serves all, and a wave's LDS accesses take effect in order, so no barrier
// is needed.  Empty slots write to `junk` (4 bytes per lane, never read)
// rather than branch around the store.  Entries past 64 kPre are read here.
template <int NS, int NR>
__device__ __forceinline__ void build_first(const MixArgs& p, int b, const int32_t* __restrict__ s,
                                            const float* __restrict__ alpha, const WaveCoefs& wc,
                                            unsigned char* rows, unsigned char* junk, bf16x8 (&bfr)[NS][NR], int cw,
                                            int lane) {
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
  const int my = lane & 15;  // this lane's expert within the wave
  const int g = lane >> 4;
#pragma unroll
  for (int q = 0; q < NR; ++q)  // 16 rows of 64 NR bytes: NR chunks per lane
    reinterpret_cast<u32x4*>(rows)[lane + 64 * q] = u32x4{0u, 0u, 0u, 0u};
  unsigned char* dst[kPre];
  uint16_t pt[kPre][NS];
#pragma unroll
  for (int r = 0; r < kPre; ++r) {
    const uint32_t sl = half_of(wc.slot[r >> 1], r);
    dst[r] = sl != 0xffffu ? rows + sl : junk + 4 * lane;
    split_parts<NS>(wc.a[r], pt[r]);
  }
  unsigned char* udst[kUPer];
#pragma unroll
  for (int u = 0; u < kUPer; ++u) {
    const uint32_t sl = half_of(wc.uslot[u >> 1], u);
    udst[u] = sl != 0xffffu ? rows + sl : junk + 4 * lane;
  }
  uint16_t ipt[NS];
  split_parts<NS>(p.nU > 0 ? 1.f / (float)p.nU : 0.f, ipt);
#pragma unroll
  for (int part = 0; part < NS; ++part) {
#pragma unroll
    for (int r = 0; r < kPre; ++r) *reinterpret_cast<uint16_t*>(dst[r]) = pt[r][part];
    for (int i = lane + 64 * kPre; i < kExpertsPerWave * p.k; i += 64) {
      const int e = kExpertsPerWave * cw * p.k + i;
      if (e < nent) *reinterpret_cast<uint16_t*>(rows + stage_off<NR>(i / p.k, s[e])) = coef_part(ab[e], part);
    }
#pragma unroll
    for (int u = 0; u < kUPer; ++u) *reinterpret_cast<uint16_t*>(udst[u]) = ipt[part];
#pragma unroll
    for (int ks = 0; ks < NR; ++ks)
      bfr[part][ks] =
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(rows + stage_off<NR>(my, 32 * ks + 8 * g)));
  }
}

// Rebuilds a consumer wave's rows of A_b when the image changes, through its
// own staging rows, 8 at a time (the ring is in use then).  For each group of
// 8 rows: zero them, then per part scatter part `part` of the coefficients
// (and 1/nU at the uncovered channels) and read the MFMA B operands of the
// lanes whose expert is in the group.
template <int NS, int NR>
__device__ __forceinline__ void build_coefs(const MixArgs& p, int b, const int32_t* __restrict__ s,
                                            const float* __restrict__ alpha, const WaveCoefs& wc,
                                            unsigned char* rows, bf16x8 (&bfr)[NS][NR], int cw, int lane) {
  constexpr int kGroupBytes = kStageRows * 64 * NR;  // 8 rows of 2 C bytes
  const int nent = p.R * p.k;
  const float* ab = alpha + (int64_t)b * nent;
  const float inv = p.nU > 0 ? 1.f / (float)p.nU : 0.f;
  const int my = lane & 15;  // this lane's expert within the wave
  const int g = lane >> 4;
#pragma unroll 1
  for (int grp = 0; grp < kExpertsPerWave / kStageRows; ++grp) {
#pragma unroll
    for (int q = 0; q < NR / 2 + (NR & 1); ++q)  // 8 rows of 64 NR bytes: 32 NR chunks
      if (lane + 64 * q < 32 * NR) reinterpret_cast<u32x4*>(rows)[lane + 64 * q] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int part = 0; part < NS; ++part) {
#pragma unroll
      for (int r = 0; r < kPre; ++r) {
        const uint32_t sl = half_of(wc.slot[r >> 1], r);
        if (sl != 0xffffu && ((int)sl >= kGroupBytes) == (grp == 1))
          *reinterpret_cast<uint16_t*>(rows + sl - grp * kGroupBytes) = coef_part(wc.a[r], part);
      }
      for (int i = lane + 64 * kPre; i < kExpertsPerWave * p.k; i += 64) {
        const int e = kExpertsPerWave * cw * p.k + i;
        const int eo = i / p.k;
        if (e < nent && (eo >> 3) == grp)
          *reinterpret_cast<uint16_t*>(rows + stage_off<NR>(eo & (kStageRows - 1), s[e])) = coef_part(ab[e], part);
      }
#pragma unroll
      for (int u = 0; u < kUPer; ++u) {
        const uint32_t sl = half_of(wc.uslot[u >> 1], u);
        if (sl != 0xffffu && ((int)sl >= kGroupBytes) == (grp == 1))
          *reinterpret_cast<uint16_t*>(rows + sl - grp * kGroupBytes) = coef_part(inv, part);
      }
#pragma unroll
      for (int ks = 0; ks < NR; ++ks) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(rows + stage_off<NR>(my & (kStageRows - 1), 32 * ks + 8 * g));
        if ((my >> 3) == grp) bfr[part][ks] = __builtin_bit_cast(bf16x8, v);
      }
    }
  }
}

__device__ __forceinline__ bf16x4 tr_read(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MOCE_LDS bf16x4*)(MOCE_LDS unsigned char*)p);
}

// Waits until the copies of tile n + 1 are complete, given that the copies
// of tiles up to min(n + 3, t1 - 1) have been issued (2 NR per tile).
template <int NR>
__device__ __forceinline__ void wait_next_tile(int n, int t1) {
  const int ahead = min(2, t1 - 2 - n);  // tiles issued after tile n + 1
  if (ahead >= 2)
    __builtin_amdgcn_s_waitcnt(vm_wait(4 * NR));
  else if (ahead == 1)
    __builtin_amdgcn_s_waitcnt(vm_wait(2 * NR));
  else
    __builtin_amdgcn_s_waitcnt(vm_wait(0));
}

// ---- one workgroup's pass over the tiles [t0, t1) -------------------------
//
// The three roles run separate loops (so that the registers one of them
// needs never constrain another) with the same barrier sequence: the
// prologue's barrier, at the first tile a barrier once tile t0 is in LDS, and
// one barrier at the end of every tile.
struct Run {
  MixArgs p;
  int t0, t1;          // tiles b * nt + j of the pass
  int tid, lane, wv;
  int tileb;           // bytes of one LDS tile buffer
  unsigned char* ring;   // kRing tile buffers
  unsigned char* stage;  // the consumer waves' staging rows
  unsigned char* obuf;   // two output buffers of kConsumers * kOutWave bytes
};

__device__ __forceinline__ Run make_run(const MixArgs& p, int t0, int t1, unsigned char* smem) {
  Run r;
  r.p = p;
  r.t0 = t0;
  r.t1 = t1;
  r.tid = threadIdx.x;
  r.lane = r.tid & 63;
  r.wv = __builtin_amdgcn_readfirstlane(r.tid >> 6);
  r.tileb = p.C * kRow;
  r.ring = smem;
  r.stage = smem + kRing * r.tileb;
  r.obuf = r.stage + kConsumers * kStageRows * p.C * 2;
  return r;
}

__device__ __forceinline__ unsigned char* out_buffer(const Run& r, int n) {
  return r.obuf + ((n - r.t0) & 1) * (kConsumers * kOutWave);
}

// Consumer waves: the support indices and the coefficients of the first
// image arrive before the prologue's barrier (one round trip); the staging
// slots are computed after it, while the loaders request the next tiles (with
// the gate inside, while the descriptor gather is in flight, before it).  The
// wave's rows of A_b are built at the first tile and rebuilt at every image
// change.
template <int NR, int NS, bool GATE>
__device__ __forceinline__ void consumer_run(const Run& r, const int32_t* __restrict__ s,
                                             const int32_t* __restrict__ U, const float* __restrict__ alpha,
                                             const GateArgs& ga) {
  const MixArgs& p = r.p;
  const int lane = r.lane, cw = r.wv;
  const int g = lane >> 4, sl = lane & 15;
  int b = r.t0 / p.nt, j = r.t0 - b * p.nt;
  WaveCoefs wc;
  unsigned char* rows = r.stage + cw * (kStageRows * 64 * NR);
  int cs[kPre], cu[kUPer];
  WaveGate wg;
  float dv[kPre];
  if constexpr (GATE)
    load_gate(p, ga, wg, cw, lane);
  else
    fetch_coefs(p, alpha, b, wc, cw, lane);
  load_indices(p, s, U, cs, cu, cw, lane);
#pragma unroll
  for (int q = 0; q < kPre; ++q) asm volatile("" : "+v"(cs[q]));
#pragma unroll
  for (int q = 0; q < kUPer; ++q) asm volatile("" : "+v"(cu[q]));
  if constexpr (GATE) {
    // the descriptors at the support entries: a second round trip, before
    // the barrier too, with the slot arithmetic done while it is in flight
    gather_desc(p, ga, b, cs, dv);
    wave_slots<NR>(p, cs, cu, wc, cw, lane);
#pragma unroll
    for (int q = 0; q < kPre; ++q) asm volatile("" : "+v"(dv[q]));
  }
  __builtin_amdgcn_s_waitcnt(vm_wait(0));
  lds_barrier();
  if constexpr (GATE)
    wave_gate(p, wg, dv, wc, cw, lane);
  else
    wave_slots<NR>(p, cs, cu, wc, cw, lane);

  // transposing reads: 16-lane group g reads channels 8 g + 4 h + (l >> 2)
  // (+ 32 ks) at positions 16 pb + 4 (l & 3) .. +3, l = lane & 15
  const int trow = (8 * g + (sl >> 2)) * kRow + 8 * (sl & 1);
  int troff[4];
#pragma unroll
  for (int pb = 0; pb < 4; ++pb) troff[pb] = trow + (((2 * pb + ((sl & 3) >> 1)) ^ tile_swz(8 * g + (sl >> 2))) << 4);
  // results: row sl of the wave's block, bytes 32 pb + 8 g (chunk 2 pb +
  // (g >> 1) before the row's swizzle)
  const int cres = cw * kOutWave + sl * kRow + 8 * (g & 1);
  // the output epilogue's constants of this lane's expert
  const bool epi = epi_active(p.ep);
  const int eo = min(kExpertsPerWave * cw + sl, p.E - 1);
  const float esc = p.ep.scale ? p.ep.scale[eo] : 1.f, esh = p.ep.scale ? p.ep.shift[eo] : 0.f;

  bf16x8 bfr[NS][NR];
  // the first build stages in the last ring buffer (4 x 16 rows of 2 C bytes)
  // and sends empty slots to this wave's own staging rows, unused until an
  // image changes
  build_first<NS, NR>(p, b, s, alpha, wc, r.ring + (kRing - 1) * r.tileb + cw * (kExpertsPerWave * 64 * NR), rows,
                      bfr, cw, lane);
  lds_barrier();  // tile t0 in LDS
  for (int n = r.t0; n < r.t1; ++n, ++j) {
    if (j == p.nt) {
      ++b;
      j = 0;
    }
    if (n != r.t0 && j == 0) {
      // next image: rebuild this wave's rows of A_b.  The old operands are
      // dead from here (each lane's are rewritten by one of the build's
      // passes); a constant frees their registers meanwhile.
#pragma unroll
      for (int part = 0; part < NS; ++part)
#pragma unroll
        for (int ks = 0; ks < NR; ++ks) bfr[part][ks] = bf16x8{};
      if constexpr (GATE) {
        // the static reads are repeated here: an opaque lane index keeps
        // them from being hoisted out of the loop, where they would stay
        // live through the products
        int ln = lane;
        asm volatile("" : "+v"(ln));
        WaveGate wg2;
        int cs2[kPre];
        float dv2[kPre];
        load_gate(p, ga, wg2, cw, ln);
#pragma unroll
        for (int q = 0; q < kPre; ++q) cs2[q] = s[min(kExpertsPerWave * cw * p.k + ln + 64 * q, p.R * p.k - 1)];
#pragma unroll
        for (int q = 0; q < kPre; ++q) asm volatile("" : "+v"(cs2[q]));
        gather_desc(p, ga, b, cs2, dv2);
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
        wave_gate(p, wg2, dv2, wc, cw, ln);
      } else {
        fetch_coefs(p, alpha, b, wc, cw, lane);
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
      }
      build_coefs<NS, NR>(p, b, s, alpha, wc, rows, bfr, cw, lane);
    }

    const unsigned char* tb = r.ring + ((n - r.t0) & (kRing - 1)) * r.tileb;
    // software pipeline: the operands of channel step ks + 1 are read while
    // the 4 NS products of step ks run, ordered so that consecutive products
    // update different accumulators
    auto read_step = [&](int ks, bf16x8 (&xa)[4]) __attribute__((always_inline)) {
#pragma unroll
      for (int pb = 0; pb < 4; ++pb) {
        const unsigned char* ap = tb + troff[pb] + ks * 32 * kRow;
        xa[pb] = __builtin_shufflevector(tr_read(ap), tr_read(ap + 4 * kRow), 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    f32x4 acc[4];
#pragma unroll
    for (int pb = 0; pb < 4; ++pb) acc[pb] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 xa[2][4];
    read_step(0, xa[0]);
#pragma unroll
    for (int ks = 0; ks < NR; ++ks) {
      if (ks + 1 < NR) read_step(ks + 1, xa[(ks + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int part = 0; part < NS; ++part)
#pragma unroll
        for (int pb = 0; pb < 4; ++pb)
          acc[pb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[ks & 1][pb], bfr[part][ks], acc[pb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    unsigned char* ob = out_buffer(r, n) + cres;
    if (epi) {
#pragma unroll
      for (int pb = 0; pb < 4; ++pb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float v = p.ep.scale ? __builtin_fmaf(acc[pb][q], esc, esh) : acc[pb][q];
          acc[pb][q] = p.ep.relu ? fmaxf(v, 0.f) : v;
        }
    }
#pragma unroll
    for (int pb = 0; pb < 4; ++pb)
      *reinterpret_cast<u32x2*>(ob + (((2 * pb + (g >> 1)) ^ (sl & 7)) << 4)) =
          u32x2{pack_bf16x2(acc[pb][0], acc[pb][1]), pack_bf16x2(acc[pb][2], acc[pb][3])};
    lds_barrier();  // results of tile n visible; reads of tile n done
  }
}

// Loader waves: the first tiles are requested after the prologue's barrier,
// once the consumers' index and descriptor reads are back (with every
// workgroup starting at once, tiles requested earlier queue those small
// reads behind megabytes of x; the consumers' gate and first build still
// take longer than tile t0's round trip), then up to three tiles stay in
// flight.
template <int NR>
__device__ __forceinline__ void loader_run(const Run& r, const uint16_t* __restrict__ x) {
  const MixArgs& p = r.p;
  const int lt = r.tid - kCThreads;
  lds_barrier();
  copy_tile<NR>(p, x, r.t0, r.ring, lt);
  if (r.t0 + 1 < r.t1) copy_tile<NR>(p, x, r.t0 + 1, r.ring + r.tileb, lt);
  if (r.t0 + 2 < r.t1) copy_tile<NR>(p, x, r.t0 + 2, r.ring + 2 * r.tileb, lt);
  for (int n = r.t0; n < r.t1; ++n) {
    if (n == r.t0) {
      wait_next_tile<NR>(r.t0 - 1, r.t1);  // tile t0 complete
      lds_barrier();
    }
    // tile n + 3 into the buffer tile n - 1 left (free since the last
    // barrier), then wait until tile n + 1 is complete
    if (n + 3 < r.t1) copy_tile<NR>(p, x, n + 3, r.ring + ((n - r.t0 + 3) & (kRing - 1)) * r.tileb, lt);
    wait_next_tile<NR>(n, r.t1);
    lds_barrier();  // tile n + 1 complete and visible
  }
}

// Store waves: the results of each tile go out during the next tile's step,
// the last tile's after the loop.
__device__ __forceinline__ void store_run(const Run& r, uint16_t* __restrict__ y) {
  const MixArgs& p = r.p;
  const int lane = r.lane;
  const int sw = r.wv - kConsumers - kLoaders;
  int b = r.t0 / p.nt, j = r.t0 - b * p.nt;
  lds_barrier();

  // results of tile (pimg, pj) from its output buffer: lane i of store wave w
  // writes physical chunk i & 7 of rows 8 h + (i >> 3) of consumer blocks
  // 2 w and 2 w + 1
  int pimg = b, pj = j;
  auto store_results = [&](const unsigned char* ob) __attribute__((always_inline)) {
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int rr = 8 * h + (lane >> 3);
        const int blk = 2 * sw + c2;
        const u32x4 v = *reinterpret_cast<const u32x4*>(ob + blk * kOutWave + rr * kRow + (lane & 7) * 16);
        const int o = kExpertsPerWave * blk + rr;
        const int pos = pj * kTile + 8 * ((lane & 7) ^ (rr & 7));
        // y is written once and not read back here: non-temporal stores keep
        // it from displacing x in the caches
        if (o < p.E && pos < p.HW)
          __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(y + ((int64_t)pimg * p.E + o) * p.HW + pos));
      }
  };

  for (int n = r.t0; n < r.t1; ++n, ++j) {
    if (j == p.nt) {
      ++b;
      j = 0;
    }
    if (n == r.t0) lds_barrier();  // tile t0 in LDS
    if (n > r.t0) store_results(out_buffer(r, n - 1));
    pimg = b;
    pj = j;
    lds_barrier();  // results of tile n visible
  }
  store_results(out_buffer(r, r.t1 - 1));
}

template <int NR, int NS, bool GATE>
__device__ __forceinline__ void run_tiles(const Run& r, const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                          const int32_t* __restrict__ s, const int32_t* __restrict__ U,
                                          const float* __restrict__ alpha, const GateArgs& ga) {
  if (r.wv < kConsumers)
    consumer_run<NR, NS, GATE>(r, s, U, alpha, ga);
  else if (r.wv < kConsumers + kLoaders)
    loader_run<NR>(r, x);
  else
    store_run(r, y);
}

// NR = C / 32 channel steps of 32, NS coefficient parts.  One contiguous
// range of tiles per workgroup.  GATE: the consumer waves evaluate the
// softplus-linear gate for their own coefficients (k = 32) from the pooled
// descriptors instead of reading alpha.
template <int NR, int NS, bool GATE>
__global__ void __launch_bounds__(kThreads, 1)
k_mfmamix(MixArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, const int32_t* __restrict__ s,
          const float* __restrict__ alpha, const int32_t* __restrict__ U, GateArgs ga) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int t0 = (int)((int64_t)blockIdx.x * p.ntiles / gridDim.x);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * p.ntiles / gridDim.x);
  if (t0 >= t1) return;
  const Run r = make_run(p, t0, t1, smem);
  run_tiles<NR, NS, GATE>(r, x, y, s, U, alpha, ga);
}

using MfmaKernel = void (*)(MixArgs, const uint16_t*, uint16_t*, const int32_t*, const float*, const int32_t*,
                            GateArgs);

template <int NS, bool GATE>
MfmaKernel pick(int nr) {
  static const MfmaKernel k[8] = {k_mfmamix<1, NS, GATE>, k_mfmamix<2, NS, GATE>, k_mfmamix<3, NS, GATE>,
                                  k_mfmamix<4, NS, GATE>, k_mfmamix<5, NS, GATE>, k_mfmamix<6, NS, GATE>,
                                  k_mfmamix<7, NS, GATE>, k_mfmamix<8, NS, GATE>};
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

namespace {

MixArgs mix_args(const Shape& sh, int nU) {
  MixArgs p;
  p.C = (int)sh.C;
  p.HW = (int)sh.HW;
  p.E = sh.E;
  p.R = sh.R;
  p.k = sh.k;
  p.nU = nU;
  p.nt = (int)((sh.HW + kTile - 1) / kTile);
  p.ntiles = (int)(sh.B * p.nt);
  return p;
}

int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  return cus;
}

}  // namespace

namespace {

hipError_t launch_mix_kernel(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                             int nU, const GateArgs* ga, void* y, hipStream_t st, const Epi& ep) {
  MixArgs p = mix_args(sh, nU);
  p.ep = ep;
  if (p.ntiles == 0) return hipSuccess;
  const int grid = std::min(cu_count(), p.ntiles);
  const size_t lds = mfma_lds(p.C);
  const MfmaKernel k = ga ? pick<kParts, true>(p.C / 32) : pick<kParts, false>(p.C / 32);
  // the dynamic LDS limit, set on the current device at every launch (the
  // library keeps no state between calls)
  const hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, st, p, static_cast<const uint16_t*>(x),
                     static_cast<uint16_t*>(y), s, alpha, U, ga ? *ga : GateArgs{});
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mfmamix(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                          int nU, void* y, hipStream_t st, const Epi& ep) {
  return launch_mix_kernel(sh, x, s, alpha, U, nU, nullptr, y, st, ep);
}

bool mfmamix_gate_fusable(const Shape& sh, int gate_kind) {
  return mfmamix_eligible(sh) && gate_kind == MOCE_GATE_SOFTPLUS_LINEAR && sh.k == 32;
}

hipError_t launch_mfmamix_gated(const Shape& sh, const void* x, const int32_t* s, const float* w, const float* d,
                                const float* a, const float* c, const int32_t* U, int nU, void* y, hipStream_t st, const Epi& ep) {
  const GateArgs ga{d, w, a, c};
  return launch_mix_kernel(sh, x, s, nullptr, U, nU, &ga, y, st, ep);
}

}  // namespace moce

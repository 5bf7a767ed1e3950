// Channels-last mixing as a dense product on the matrix cores, driven by a
// channel schedule of the static supports (Sec. 3.2: the supports are fixed at
// inference, so where every coefficient lands can be worked out ahead of the
// products).
//
// For one image b the routed outputs (Sec. 3.3 Eq. 5) and the residual output
// (Sec. 3.4 Eq. 6) are y_b = A_b x_b, with row o < E-1 of A_b holding
// alpha[b][o][i] at column s[o][i] and row E-1 holding 1/|U| at the uncovered
// channels.  With x channels-last, a tile of positions x 64 channels is
// already the layout of the MFMA's A operand (two K slices), so this kernel
// evaluates y^T = x^T A_b^T with 16x16x32 bf16 MFMAs over 64-channel steps, positions
// as M and experts as N.  A_b is 1/16 dense at the ResNet-50 stage-3/4 and
// ViT shapes; the matrix cores still run the dense product faster than the
// vector ALUs run the gather form.
//
// The schedule.  Dense A_b is never built: per 64-channel step only the
// support entries whose channel falls in the step are written into zeroed LDS
// rows of A_b^T (the B operand), and they are cleared again two steps later,
// before the next entries go into the same buffer.  A small kernel (k_sched)
// buckets the entries by step once per forward, one bucket per builder wave
// of a mix workgroup, each entry carrying the LDS byte offset of its slot.
//
// Exactness.  x is bf16; each float32 coefficient is split into NS bf16 parts
// (hi, the rounded remainder, and with NS = 3 the remainder of that), one
// MFMA per part, accumulated in float32.  Three parts sum to the coefficient
// exactly; two carry it to 16 significant bits (relative error at most 2^-17,
// 2^8 below the rounding of the bf16 output).
//
// Work split.  A workgroup takes MT = 16 MB positions of one image and
// NE = 64 NB consecutive experts (4 NB groups of 16) and walks the C/32
// channel steps with three kinds of waves meeting at one barrier per step:
//  - four consumer waves: wave w owns N blocks NB w .. NB w + NB - 1 and all
//    MT positions, and only issues LDS reads and MFMAs;
//  - eight builder waves: builder j owns the expert groups j and j + 8 of the
//    range and writes their B rows: at step ks it clears its entries of step
//    ks - 1 and writes those of step ks + 1 (in the buffer the consumers left
//    at the barrier).  Each builder owns whole rows, so no two waves ever
//    touch one slot.  The schedule is prefetched several steps ahead into
//    registers, and the bucket's offsets sit in registers, so a step never
//    waits on memory; eight waves (two per SIMD) keep the dependent chains of
//    the coefficient arithmetic overlapped;
//  - two loader waves: copy 64-channel chunks of the x tile straight into a
//    ring of LDS buffers with global-to-LDS loads, several chunks in flight.
// At the end the consumers stage their results in LDS and every wave writes
// whole rows of y.
//
// Channels-first x (NCHW) takes the same schedule and builders with the roles
// of the operands exchanged: y_b = A_b x_b with A_b's rows (the B buffers
// above, experts by channels) as the MFMA's A operand and the x tile as its B
// operand.  The tile holds one row of MT positions per channel, copied 4 bytes
// a lane by four loader waves (channel rows start only 8-byte aligned when H W
// is a multiple of 4); the consumers read its columns with the transposing LDS
// read, and the results are staged expert by expert and written as rows of
// positions.  Each row is rotated by 64 bytes per group of 8 channels, so the
// 16 rows one transposing read touches fall on distinct banks.
#include <algorithm>
#include <utility>

#include "moce_internal.h"
#include "pool_rows.h"

namespace moce {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
#define GMIX_LDS __attribute__((address_space(3)))

constexpr int kStep = 64;                 // channels per step: two K slices of the MFMA, one x chunk
constexpr int kXRow = kStep * 2;          // bytes of one position row of an x chunk
constexpr int kBRow = kStep * 2;          // bytes of one expert row of one part of a B buffer
constexpr int kMaxXRing = 8;              // x chunk buffers at most (the ring fills the LDS left over)
constexpr int kConsumers = 4;
constexpr int kBuilders = 8;
// loader waves: 16-byte copies of channels-last rows, 4-byte copies of
// channels-first rows
constexpr int loaders_of(bool NH) { return NH ? 2 : 4; }
constexpr int threads_of(bool NH) { return 64 * (kConsumers + kBuilders + loaders_of(NH)); }
constexpr int kGroup = 16;                // experts per group (one MFMA N block)
constexpr int kGroupsPerBuilder = 2;      // 4 NB <= 16 groups per workgroup over 8 builders
constexpr int kMaxSteps = 64;             // C <= 4096: offsets 0 .. 63 in one register, the total beside
// 64-entry rounds of a builder's step held in registers: two for one group
// of 16 experts (about 16 k 64 / C entries a step), three for two; longer
// lists take a slow path
constexpr int rounds_of(int NB) { return NB <= 2 ? 2 : 3; }
constexpr int kAhead = 4;                 // steps of schedule a builder holds in registers (even)
constexpr int kCachePolicyNT = 2;         // non-temporal bit of the global-to-LDS load
constexpr int kLdsBytes = 160 * 1024;  // per CU

// Schedule entry: x = byte offset of the coefficient's slot in one part of a
// B buffer (15 bits) | the expert's slot within the workgroup's expert range
// << 15 (8 bits) | residual flag << 23; y = the selected logit's bits.
constexpr uint32_t kOffMask = 0x7fff;
constexpr int kSlotShift = 15;
constexpr uint32_t kResidualFlag = 1u << 23;

// byte offset of B[o][c] (o: expert within the workgroup, c: channel within
// the step) in one part of a B buffer: 16-byte chunk c/8 of the 128-byte row
// o, stored at chunk (c/8) ^ ((o / 2) mod 8), so that 16 consecutive rows
// read at one chunk hit 16 different bank groups (the x tile's rows are
// swizzled the same way)
__host__ __device__ inline int swz(int row) { return (row >> 1) & 7; }
__host__ __device__ inline int b_off(int o, int c) {
  return o * kBRow + (((c >> 3) ^ swz(o)) << 4) + ((c & 7) << 1);
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// s_waitcnt operand: at most n vector memory operations of this wave
// outstanding (the LDS/scalar and export counters left at their maxima)
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

struct GmArgs {
  const uint16_t* x;
  uint16_t* y;
  const int32_t* off;   // [buckets][nsteps + 1]
  const uint2* ent;     // [buckets][cap]
  const float* st;      // softmax statistics, three planes of B R floats
  int64_t nst;          // B R
  int C, HW, E, R, nU;
  int nsteps, ngroups, cap;
  int nt, nq;           // position tiles per image, expert ranges per image
  int units, per;       // work units, units per XCD slot
  float inv_nU;
  Epi ep;               // output epilogue, applied to the accumulators before rounding
};

// ---------------------------------------------------------------- schedule
// Bucket (q, j) holds the entries of expert groups j and j + 8 of expert
// range q (the ng groups of one mix workgroup), the residual row E-1 included
// where it falls there, counted and placed by step.  Order within a step is
// free: every entry writes its own slot of A_b.
struct SchedArgs {
  const int32_t* s;
  const float* w;
  const int32_t* U;
  int nU, R, k, nsteps, cap, ng, ngroups, nbuckets;
  int32_t* off;
  uint2* ent;
};

// bucket `bk` by the whole workgroup (cnt, cur: LDS of kMaxSteps ints each)
__device__ __forceinline__ void sched_bucket(const SchedArgs& a, int bk, int* cnt, int* cur) {
  const int q = bk / kBuilders, j = bk % kBuilders, tid = threadIdx.x, nth = blockDim.x;
  // the bucket's groups and their entry counts
  int gid[kGroupsPerBuilder], nr[kGroupsPerBuilder], first[kGroupsPerBuilder + 1];
  first[0] = 0;
#pragma unroll
  for (int h = 0; h < kGroupsPerBuilder; ++h) {
    const int gl = j + kBuilders * h;
    gid[h] = q * a.ng + gl;
    const bool live = gl < a.ng && gid[h] < a.ngroups;
    const int o_first = gid[h] * kGroup;
    nr[h] = live ? max(0, min(kGroup, a.R - o_first)) * a.k : 0;
    const int nres = live && a.R >= o_first && a.R < o_first + kGroup ? a.nU : 0;
    first[h + 1] = first[h] + nr[h] + nres;
  }
  const int total = first[kGroupsPerBuilder];
  // entry e of the bucket: (expert, channel, logit, residual?)
  auto entry = [&](int e, int& o, int& c, float& wv, bool& res) __attribute__((always_inline)) {
    int h = 0;
#pragma unroll
    for (int t = 1; t < kGroupsPerBuilder; ++t) h += e >= first[t] ? 1 : 0;
    const int r = e - first[h];
    const int o_first = gid[h] * kGroup;
    res = r >= nr[h];
    if (!res) {
      o = o_first + r / a.k;
      c = a.s[(int64_t)o_first * a.k + r];
      wv = a.w[(int64_t)o_first * a.k + r];
    } else {
      o = a.R;
      c = a.U[r - nr[h]];
      wv = 0.f;
    }
  };
  // each thread reads kHold entries (all loads in flight) before it counts
  // or places any of them
  constexpr int kHold = 8;
  auto each = [&](auto&& f) __attribute__((always_inline)) {
    for (int e0 = tid; e0 < total; e0 += kHold * nth) {
      int o[kHold], c[kHold];
      float wv[kHold];
      bool res[kHold];
#pragma unroll
      for (int u = 0; u < kHold; ++u) {
        c[u] = -1;
        if (e0 + u * nth < total) entry(e0 + u * nth, o[u], c[u], wv[u], res[u]);
      }
#pragma unroll
      for (int u = 0; u < kHold; ++u)
        if (c[u] >= 0) f(o[u], c[u], wv[u], res[u]);
    }
  };
  for (int t = tid; t < a.nsteps; t += nth) cnt[t] = 0;
  __syncthreads();
  each([&](int, int c, float, bool) __attribute__((always_inline)) { atomicAdd(&cnt[c >> 6], 1); });
  __syncthreads();
  // exclusive scan of the counts (nsteps <= 64: one wave)
  int32_t* ob = a.off + (int64_t)bk * (a.nsteps + 1);
  if (tid < 64) {
    const int v = tid < a.nsteps ? cnt[tid] : 0;
    int incl = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(incl, d, 64);
      if (tid >= d) incl += t;
    }
    if (tid < a.nsteps) {
      cur[tid] = incl - v;
      ob[tid] = incl - v;
    }
    if (tid == 63) ob[a.nsteps] = incl;
  }
  __syncthreads();
  const int ne = a.ng * kGroup;
  uint2* eb = a.ent + (int64_t)bk * a.cap;
  each([&](int o, int c, float wv, bool res) __attribute__((always_inline)) {
    const int pos = atomicAdd(&cur[c >> 6], 1);
    const int ow = o - q * ne;  // the expert's slot within the range
    const uint32_t packed = (uint32_t)b_off(ow, c & 63) | ((uint32_t)ow << kSlotShift) | (res ? kResidualFlag : 0u);
    eb[pos] = make_uint2(packed, __float_as_uint(wv));
  });
}

// Pooling and the schedule in one launch: workgroups below nbuckets build a
// schedule bucket each, the rest pool one (image, channel block) each, so the
// schedule's latency chains run beside memory-bound work.
template <typename T>
__global__ void __launch_bounds__(kPoolThreads)
k_pool_sched(const T* __restrict__ x, float* __restrict__ d, int C, int HW, int nblk, SchedArgs a) {
  __shared__ float part[kPoolGroups * 32 * PoolVec<T>::EPV];
  if ((int)blockIdx.x < a.nbuckets) {
    int* cnt = reinterpret_cast<int*>(part);
    sched_bucket(a, blockIdx.x, cnt, cnt + kMaxSteps);
    return;
  }
  const int i = blockIdx.x - a.nbuckets;
  pool_rows_block<T>(x, d, C, HW, i / nblk, i % nblk, part, C, 1);
}

// The same for channels-first planes of a multiple of 4 positions:
// workgroups below nbuckets build a schedule bucket each, the rest pool
// planes with L lanes each (the lanes and order of the plane pooling kernel,
// so the descriptor has the same bits).
template <int L>
__global__ void __launch_bounds__(kPoolThreads)
k_pool_sched_planes(const uint16_t* __restrict__ x, float* __restrict__ d, int64_t planes, int HW, SchedArgs a) {
  if ((int)blockIdx.x < a.nbuckets) {
    __shared__ int cc[2 * kMaxSteps];
    sched_bucket(a, blockIdx.x, cc, cc + kMaxSteps);
    return;
  }
  const int64_t group = ((int64_t)(blockIdx.x - a.nbuckets) * kPoolThreads + threadIdx.x) / L;
  const int64_t ngroups = ((int64_t)(gridDim.x - a.nbuckets) * kPoolThreads) / L;
  pool_planes8<L>(x, d, planes, HW, group, ngroups);
}

// ---------------------------------------------------------------- the mix
template <int MB, int NB, int NS, int OCC, bool NH>
struct Layout {
  static constexpr int MT = 16 * MB;                 // positions per tile
  static constexpr int NE = 64 * NB;                 // experts per workgroup
  static constexpr int XBUF = MT * kXRow;            // one x chunk
  static_assert(NS == 2, "two coefficient parts");
  static constexpr int PART = (NE + 1) * kBRow;      // one part of one B buffer: NE rows and a trash row
  static constexpr int TRASH = NE * kBRow;           // the trash row, stored into by lanes with no entry
  static constexpr int BBUF = NS * PART;             // one B buffer
  // as many x chunks in flight as the LDS left by the B buffers and the
  // statistics allows (OCC workgroups per CU share its LDS): at most
  // kMaxXRing, and so that one loader wave's outstanding copies stay within
  // its 6-bit counter
  static constexpr int XR_FIT = (kLdsBytes / OCC - 1024 - 2 * BBUF - 16 * NE) / XBUF;
  // copies per loader lane per chunk: MT / 16 of 16 bytes (channels-last),
  // MT / 8 of 4 bytes (channels-first)
  static constexpr int ROUNDS = NH ? MB : 2 * MB;
  static constexpr int XR_CNT = 63 / ROUNDS + 1;
  static constexpr int XR = XR_FIT < kMaxXRing ? (XR_FIT < XR_CNT ? XR_FIT : XR_CNT)
                                               : (kMaxXRing < XR_CNT ? kMaxXRing : XR_CNT);
  static_assert(XR >= 2, "at least two x chunk buffers");
  static constexpr int OFF_X = 0;
  static constexpr int OFF_B = OFF_X + XR * XBUF;
  static constexpr int OFF_ST = OFF_B + 2 * BBUF;    // statistics, one float4 (rt, m, rzs, -) per expert
  // staging rows of the results: one per position (channels-last) or per
  // expert (channels-first)
  static constexpr int OROW = NH ? NE * 2 + 16 : MT * 2 + 16;
  static size_t bytes() {
    const size_t main = (size_t)OFF_ST + (size_t)16 * NE;
    const size_t stage = (size_t)(NH ? MT : NE) * OROW;
    return std::max(main, stage);
  }
  // channels-first x chunk: channel row r's byte u (positions u / 2) at
  // r ROWB + (u + rot(r)) mod ROWB
  static constexpr int ROWB = MT * 2;
  __device__ static int rot(int r) { return (64 * ((r >> 3) & 3)) % ROWB; }
};

// the exact split of a float into bf16 parts (hi, the rounded remainder, ...)
template <int NS>
__device__ __forceinline__ void split_parts(float a, uint16_t (&pt)[NS]) {
  pt[0] = f32_to_bf16(a);
  if constexpr (NS > 1) {
    const float r1 = a - bf16_to_f32(pt[0]);
    pt[1] = f32_to_bf16(r1);
    if constexpr (NS > 2) pt[2] = f32_to_bf16(r1 - bf16_to_f32(pt[1]));
  }
}

// work unit of this workgroup: units of one image are consecutive, and
// consecutive units go to one XCD (workgroup u runs on XCD u mod 8), so the
// workgroups that share an image share that XCD's L2
__device__ __forceinline__ int unit_of(const GmArgs& p) {
  const int u = blockIdx.x;
  return (u & 7) * p.per + (u >> 3);
}

template <int MB, int NB, int NS, int OCC>
__device__ __forceinline__ void consumer(const GmArgs& p, unsigned char* smem, int wv, int o0) {
  using L = Layout<MB, NB, NS, OCC, true>;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, n = lane & 15;
  f32x4 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // fragments of K slice h of a step: A row 16 mb + n and B row
  // 16 (NB wv + nb) + n, logical chunk 4 h + g of the row, stored at
  // chunk (4 h + g) ^ swz(row) = (4 h + g) ^ (n >> 1)
  const int arow = n * kXRow;
  const int brow = (16 * NB * wv + n) * kBRow;
  const int ch0 = (g ^ (n >> 1)) << 4, ch1 = ((4 + g) ^ (n >> 1)) << 4;
  // A step is two K slices.  A slice runs one pass per part: every
  // accumulator once, so an accumulator's products are MB NB MFMAs apart.
  // The next slice's fragments are read into the registers of this slice's
  // as soon as their last use is issued: its B part-0 fragments after this
  // slice's part-0 pass, its A fragments block by block in the part-1 pass,
  // its B part-1 fragments after it; only the step's first slice waits for
  // its reads (the barrier before it is what makes them valid).
  auto load_a = [&](const unsigned char* xb, int h, int mb) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const u32x4*>(xb + mb * 16 * kXRow + (h ? ch1 : ch0)));
  };
  auto load_b = [&](const unsigned char* bb, int h, int nb, int pt) __attribute__((always_inline)) {
    return __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(bb + pt * L::PART + nb * 16 * kBRow + (h ? ch1 : ch0)));
  };
  lds_barrier();  // prologue: chunk 0 and the step-0 coefficients are in LDS
  for (int ks = 0; ks < p.nsteps; ++ks) {
    const unsigned char* xb = smem + L::OFF_X + (ks % L::XR) * L::XBUF + arow;
    const unsigned char* bb = smem + L::OFF_B + (ks & 1) * L::BBUF + brow;
    bf16x8 a[MB], b0[NB], b1[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b0[nb] = load_b(bb, 0, nb, 0);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) a[mb] = load_a(xb, 0, mb);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b1[nb] = load_b(bb, 0, nb, 1);
    // the compiler's scheduler would move each read next to its first use;
    // the fences keep them where they are issued here
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mb], b0[nb], acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (h == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) b0[nb] = load_b(bb, 1, nb, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mb], b1[nb], acc[mb][nb], 0, 0, 0);
        if (h == 0) {
          __builtin_amdgcn_sched_barrier(0);
          a[mb] = load_a(xb, 1, mb);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (h == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) b1[nb] = load_b(bb, 1, nb, 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    lds_barrier();  // step ks done: its x chunk and B buffer may be reused
  }
  // results: D[m][n] of block (mb, nb) sits on lane n + 16 (m / 4), element m % 4
  unsigned char* stg = smem;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * mb + 4 * g + r;
        const int col = 16 * (NB * wv + nb) + n;
        *reinterpret_cast<uint16_t*>(stg + row * L::OROW + col * 2) =
            f32_to_bf16(epi_apply(p.ep, acc[mb][nb][r], min(o0 + col, p.E - 1)));
      }
}

template <int MB, int NB, int NS, int OCC, bool NH>
__device__ __forceinline__ void builder(const GmArgs& p, unsigned char* smem, int j, int b, int q) {
  using L = Layout<MB, NB, NS, OCC, NH>;
  constexpr int NG = 4 * NB;  // groups of the range
  constexpr int kRounds = rounds_of(NB);
  const int lane = threadIdx.x & 63;
  float4* st = reinterpret_cast<float4*>(smem + L::OFF_ST);
  const int o0 = q * L::NE;
  const int bucket = q * kBuilders + j;
  const int32_t* ob = p.off + (int64_t)bucket * (p.nsteps + 1);
  const uint2* eb = p.ent + (int64_t)bucket * p.cap;
  // step 0's list starts at the bucket's first entry, so its loads go out
  // first, beside those of the offsets and the statistics: the prologue waits
  // for one round trip to memory instead of two
  uint2 e0[kRounds];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) e0[r] = eb[min(64 * r + lane, p.cap - 1)];
  // this builder's groups' statistics into LDS and their B rows (both
  // buffers, every part) zeroed; the bucket's offsets into registers
#pragma unroll
  for (int h = 0; h < kGroupsPerBuilder; ++h) {
    const int gl = j + kBuilders * h;
    if (gl >= NG) continue;
    if (lane < kGroup) {
      const int ow = kGroup * gl + lane;
      const int64_t bo = (int64_t)b * p.R + min(o0 + ow, p.R - 1);
      st[ow] = make_float4(p.st[bo], p.st[p.nst + bo], p.st[2 * p.nst + bo], 0.f);
    }
    for (int i = lane; i < 2 * NS * kGroup * (kBRow / 16); i += 64) {
      const int part = i / (kGroup * (kBRow / 16));  // buffer * NS + part
      const int r = i - part * (kGroup * (kBRow / 16));
      *reinterpret_cast<u32x4*>(smem + L::OFF_B + part * L::PART + (kGroup * gl) * kBRow + r * 16) =
          u32x4{0u, 0u, 0u, 0u};
    }
  }
  const int ofr = ob[min(lane, p.nsteps)];
  const int tot = __builtin_amdgcn_readfirstlane(ob[p.nsteps]);
  // offset t of the bucket (t uniform, 0 <= t <= nsteps <= 64)
  auto ofs = [&](int t) __attribute__((always_inline)) {
    return t < kMaxSteps ? __builtin_amdgcn_readlane(ofr, t) : tot;
  };
  // step t's entries, rounds 0 .. kRounds - 1 (t clamped into range; reads
  // past the step's list are clamped to the bucket: valid, never used)
  auto fetch = [&](int t, uint2 (&e)[kRounds]) __attribute__((always_inline)) {
    const int tc = min(t, p.nsteps - 1);
    const int beg = ofs(tc);
#pragma unroll
    for (int r = 0; r < kRounds; ++r) e[r] = eb[min(beg + 64 * r + lane, p.cap - 1)];
    return ofs(tc + 1) - beg;
  };
  __builtin_amdgcn_s_waitcnt(vm_wait(0));
  __builtin_amdgcn_s_waitcnt(0xc07f);  // this wave's LDS writes done (lgkmcnt 0)

  // a step's list into buffer `buf`: all coefficients first (a lane past the
  // end holds a placeholder, clamped into range and never stored), then the
  // stores; more than 64 kRounds entries (rare) are read one round at a time
  auto put = [&](unsigned char* buf, int t, const uint2 (&e)[kRounds], int n, bool clear)
      __attribute__((always_inline)) {
    // a lane past the list's end stores into the trash row instead of
    // branching around its store; rounds wholly past the end are skipped
    // (uniform: n is the wave's)
    int off[kRounds];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) off[r] = 64 * r + lane < n ? (int)(e[r].x & kOffMask) : L::TRASH;
    if (clear) {
#pragma unroll
      for (int r = 0; r < kRounds; ++r)
        if (r == 0 || 64 * r < n)
#pragma unroll
          for (int v = 0; v < NS; ++v) *reinterpret_cast<uint16_t*>(buf + v * L::PART + off[r]) = 0;
    } else {
      float4 sv[kRounds];
#pragma unroll
      for (int r = 0; r < kRounds; ++r)
        if (r == 0 || 64 * r < n) sv[r] = st[min((int)((e[r].x >> kSlotShift) & 0xff), L::NE - 1)];
#pragma unroll
      for (int r = 0; r < kRounds; ++r)
        if (r == 0 || 64 * r < n) {
          const float a = (e[r].x & kResidualFlag)
                              ? p.inv_nU
                              : coef_alpha(coef_e(coef_z(__uint_as_float(e[r].y), sv[r].x), sv[r].y), sv[r].z);
          uint16_t pt[NS];
          split_parts<NS>(a, pt);
#pragma unroll
          for (int v = 0; v < NS; ++v) *reinterpret_cast<uint16_t*>(buf + v * L::PART + off[r]) = pt[v];
        }
    }
    for (int q0 = 64 * kRounds; q0 < n; q0 += 64) {
      const uint2 x = eb[min(ofs(t) + q0 + lane, p.cap - 1)];
      uint16_t px[NS] = {0, 0};
      if (!clear) {
        const float4 s1 = st[min((int)((x.x >> kSlotShift) & 0xff), L::NE - 1)];
        const float a = (x.x & kResidualFlag) ? p.inv_nU
                                              : coef_alpha(coef_e(coef_z(__uint_as_float(x.y), s1.x), s1.y), s1.z);
        split_parts<NS>(a, px);
      }
      if (q0 + lane < n)
#pragma unroll
        for (int v = 0; v < NS; ++v) *reinterpret_cast<uint16_t*>(buf + v * L::PART + (x.x & kOffMask)) = px[v];
    }
  };

  // schedule ring: ring[t % kAhead] holds step t's list, cnt its length;
  // prev[t & 1] keeps step t - 2's for the clearing
  uint2 ring[kAhead][kRounds];
  int cnt[kAhead];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) ring[0][r] = e0[r];
  cnt[0] = ofs(min(1, p.nsteps)) - ofs(0);
#pragma unroll
  for (int a = 1; a < kAhead; ++a) cnt[a] = fetch(a, ring[a]);
  uint2 prev[2][kRounds];
  int pcnt[2] = {0, 0};
  __builtin_amdgcn_s_waitcnt(vm_wait((kAhead - 1) * kRounds));
  put(smem + L::OFF_B, 0, ring[0], cnt[0], false);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) prev[0][r] = ring[0][r];
  pcnt[0] = cnt[0];
  cnt[0] = fetch(kAhead, ring[0]);
  lds_barrier();  // prologue
  // step ks: consumers multiply step ks; this builder writes step ks + 1
  for (int ks0 = 0; ks0 < p.nsteps; ks0 += kAhead) {
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      const int ks = ks0 + u;
      const int t = ks + 1;
      // ks0 is a multiple of kAhead (even), so the ring slot and the parity
      // of t are constants of the unrolled body.  The ring is refilled on
      // every step, past the end too (clamped, valid reads): a refill under a
      // condition would merge the in-flight load with the old register at
      // the join, and the copy that merge needs would wait for the load
      const int slot = (u + 1) % kAhead;
      const int par = (u + 1) & 1;
      __builtin_amdgcn_s_waitcnt(vm_wait((kAhead - 1) * kRounds));
      if (t < p.nsteps) {
        unsigned char* buf = smem + L::OFF_B + (t & 1) * L::BBUF;
        if (t >= 2) put(buf, t - 2, prev[par], pcnt[par], true);
        put(buf, t, ring[slot], cnt[slot], false);
      }
#pragma unroll
      for (int r = 0; r < kRounds; ++r) prev[par][r] = ring[slot][r];
      pcnt[par] = cnt[slot];
      cnt[slot] = fetch(t + kAhead, ring[slot]);
      if (ks < p.nsteps) lds_barrier();
    }
  }
}

// waits until at most n chunk copies of this loader wave are outstanding
// (n < XR; one s_waitcnt with a constant operand per possible n)
template <int ROUNDS, int... Cs>
__device__ __forceinline__ void wait_chunks_of(int n, std::integer_sequence<int, Cs...>) {
  ((n == Cs ? (__builtin_amdgcn_s_waitcnt(vm_wait(Cs * ROUNDS)), 0) : 0), ...);
}
template <int ROUNDS, int XR>
__device__ __forceinline__ void wait_chunks(int n) {
  static_assert((XR - 1) * ROUNDS <= 63, "outstanding copies fit the counter");
  wait_chunks_of<ROUNDS>(n, std::make_integer_sequence<int, XR>{});
}

template <int MB, int NB, int NS, int OCC>
__device__ __forceinline__ void loader(const GmArgs& p, unsigned char* smem, int lw, int b, int p0) {
  using L = Layout<MB, NB, NS, OCC, true>;
  constexpr int XR = L::XR;
  const int lane = threadIdx.x & 63;
  const int nchunks = p.nsteps;
  // chunk n (the x tile's channels of step n) into ring slot n % XR.  Global
  // round u = 2 r + lw of the chunk (rounds r of this loader wave) covers
  // slots 64 u .. 64 u + 63: row (64 u + l) / 8, stored chunk l % 8 holding
  // logical chunk (l % 8) ^ swz(row); rows past the image repeat its last row
  auto copy = [&](int n) __attribute__((always_inline)) {
    GMIX_LDS unsigned char* dst = (GMIX_LDS unsigned char*)(smem + L::OFF_X + (n % XR) * L::XBUF);
#pragma unroll
    for (int r = 0; r < L::ROUNDS; ++r) {
      const int u = 2 * r + lw;
      const int row = 8 * u + (lane >> 3);
      const int pos = min(p0 + row, p.HW - 1);
      const int logical = (lane & 7) ^ swz(row);
      const uint16_t* src = p.x + ((int64_t)b * p.HW + pos) * p.C + n * kStep + logical * 8;
      __builtin_amdgcn_global_load_lds((const void*)src, (GMIX_LDS void*)(dst + u * 1024), 16, 0, kCachePolicyNT);
    }
  };
  // prologue: chunk 0 complete; chunks 1 .. XR - 2 go out after the barrier
  copy(0);
  wait_chunks<L::ROUNDS, XR>(0);
  lds_barrier();  // prologue
  for (int n = 1; n < min(XR - 1, nchunks); ++n) copy(n);
  for (int ks = 0; ks < p.nsteps; ++ks) {
    // chunk ks + XR - 1 into the slot chunk ks - 1 left (free since the
    // barrier that ended step ks - 1); chunk ks + 1 complete before this
    // step's barrier, the later ones may fly on
    if (ks + XR - 1 < nchunks) copy(ks + XR - 1);
    if (ks + 1 < nchunks) wait_chunks<L::ROUNDS, XR>(min(ks + XR - 1, nchunks - 1) - (ks + 1));
    lds_barrier();
  }
}


// Channels-first consumer: D[e][p] = A_b[e][:] x[:][p] with A = the B
// buffers' expert rows, B = the x tile's columns through the transposing read.
// Wave wv owns expert blocks NB wv .. NB wv + NB - 1 and all MT positions.
template <int MB, int NB, int NS, int OCC>
__device__ __forceinline__ void consumer_t(const GmArgs& p, unsigned char* smem, int wv, int o0) {
  using L = Layout<MB, NB, NS, OCC, false>;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, n = lane & 15;
  f32x4 acc[NB][MB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // A fragments: expert row 16 (NB wv + nb) + n, logical chunk 4 h + g
  const int brow = (16 * NB * wv + n) * kBRow;
  const int ch0 = (g ^ (n >> 1)) << 4, ch1 = ((4 + g) ^ (n >> 1)) << 4;
  auto load_c = [&](const unsigned char* bb, int h, int nb, int pt) __attribute__((always_inline)) {
    return __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(bb + pt * L::PART + nb * 16 * kBRow + (h ? ch1 : ch0)));
  };
  // B fragments of K slice h, position block mb: lane j of 16-lane group G
  // takes channels 32 h + 8 G .. + 7 at position 16 mb + j.  In each
  // transposing read source lane 4 t + q of the group addresses channel row
  // 32 h + 8 G + t (then + 4) at positions 16 mb + 4 q .. + 3; all of this
  // lane's rows share the rotation of group G
  const int t = (lane >> 2) & 3, q = lane & 3;
  const int r0 = 8 * g + t;
  const int ub = 8 * q + L::rot(r0);
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  auto load_x = [&](const unsigned char* xb, int h, int mb) __attribute__((always_inline)) {
    int u = ub + 32 * mb;
    u = u >= L::ROWB ? u - L::ROWB : u;
    const unsigned char* a0 = xb + (32 * h + r0) * L::ROWB + u;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a0);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a0 + 4 * L::ROWB));
    const s16x8 v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    return __builtin_bit_cast(bf16x8, v);
  };
  lds_barrier();  // prologue: chunk 0 and the step-0 coefficients are in LDS
  for (int ks = 0; ks < p.nsteps; ++ks) {
    const unsigned char* xb = smem + L::OFF_X + (ks % L::XR) * L::XBUF;
    const unsigned char* bb = smem + L::OFF_B + (ks & 1) * L::BBUF + brow;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // the slice's A fragments, then its x fragments one position block at
      // a time, each read one block ahead of its products
      bf16x8 c0[NB], c1[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        c0[nb] = load_c(bb, h, nb, 0);
        c1[nb] = load_c(bb, h, nb, 1);
      }
      bf16x8 xv = load_x(xb, h, 0);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 xn = load_x(xb, h, mb + 1 < MB ? mb + 1 : mb);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c0[nb], xv, acc[nb][mb], 0, 0, 0);
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c1[nb], xv, acc[nb][mb], 0, 0, 0);
        }
        xv = xn;
      }
    }
    lds_barrier();  // step ks done: its x chunk and B buffer may be reused
  }
  // results: D[e][p] of block (nb, mb) sits on lane p + 16 (e / 4), element
  // e % 4; staged as rows of positions, one per expert
  unsigned char* stg = smem;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * (NB * wv + nb) + 4 * g + r;
        const int col = 16 * mb + n;
        *reinterpret_cast<uint16_t*>(stg + row * L::OROW + col * 2) =
            f32_to_bf16(epi_apply(p.ep, acc[nb][mb][r], min(o0 + row, p.E - 1)));
      }
}

// Channels-first loader: chunk n is channels 64 n .. 64 n + 63 of the tile,
// one rotated row of MT positions each, copied 4 bytes a lane.  Copy i of a
// chunk fills LDS bytes 256 i .. 256 i + 255; loader wave lw issues copies
// lw, lw + 4, ...  Positions past the image load its last two positions.
template <int MB, int NB, int NS, int OCC>
__device__ __forceinline__ void loader_t(const GmArgs& p, unsigned char* smem, int lw, int b, int p0) {
  using L = Layout<MB, NB, NS, OCC, false>;
  constexpr int XR = L::XR;
  constexpr int NL = loaders_of(false);
  const int lane = threadIdx.x & 63;
  const int nchunks = p.nsteps;
  // this lane's source offsets (elements from the chunk's first channel row)
  int src[L::ROUNDS];
#pragma unroll
  for (int r = 0; r < L::ROUNDS; ++r) {
    const int o = 256 * (lw + NL * r) + 4 * lane;
    const int row = o / L::ROWB;
    int u = o - row * L::ROWB - L::rot(row);
    if (u < 0) u += L::ROWB;
    const int pos = min(p0 + u / 2, p.HW - 2);
    src[r] = row * p.HW + pos;
  }
  const uint16_t* xb = p.x + (int64_t)b * p.C * p.HW;
  auto copy = [&](int n) __attribute__((always_inline)) {
    GMIX_LDS unsigned char* dst = (GMIX_LDS unsigned char*)(smem + L::OFF_X + (n % XR) * L::XBUF);
    const uint16_t* cb = xb + (int64_t)n * kStep * p.HW;
#pragma unroll
    for (int r = 0; r < L::ROUNDS; ++r)
      __builtin_amdgcn_global_load_lds((const void*)(cb + src[r]), (GMIX_LDS void*)(dst + 256 * (lw + NL * r)), 4,
                                       0, kCachePolicyNT);
  };
  const int first = min(XR - 1, nchunks);
  for (int n = 0; n < first; ++n) copy(n);
  wait_chunks<L::ROUNDS, XR>(first - 1);
  lds_barrier();  // prologue
  for (int ks = 0; ks < p.nsteps; ++ks) {
    if (ks + XR - 1 < nchunks) copy(ks + XR - 1);
    if (ks + 1 < nchunks) wait_chunks<L::ROUNDS, XR>(min(ks + XR - 1, nchunks - 1) - (ks + 1));
    lds_barrier();
  }
}

template <int MB, int NB, int NS, int OCC, bool NH>
__global__ void __launch_bounds__(threads_of(NH), OCC)
k_gmix(GmArgs p) {
  using L = Layout<MB, NB, NS, OCC, NH>;
  constexpr int kThreads = threads_of(NH);
  extern __shared__ __align__(16) unsigned char smem[];
  const int v = unit_of(p);
  if (v >= p.units) return;  // uniform per workgroup: no barrier is skipped by part of it
  const int per_img = p.nt * p.nq;
  const int b = v / per_img;
  const int r = v - b * per_img;
  const int jt = r / p.nq, q = r - (r / p.nq) * p.nq;
  const int p0 = jt * L::MT, o0 = q * L::NE;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (wv < kConsumers) {
    if constexpr (NH)
      consumer<MB, NB, NS, OCC>(p, smem, wv, o0);
    else
      consumer_t<MB, NB, NS, OCC>(p, smem, wv, o0);
  } else if (wv < kConsumers + kBuilders) {
    builder<MB, NB, NS, OCC, NH>(p, smem, wv - kConsumers, b, q);
  } else {
    if constexpr (NH)
      loader<MB, NB, NS, OCC>(p, smem, wv - kConsumers - kBuilders, b, p0);
    else
      loader_t<MB, NB, NS, OCC>(p, smem, wv - kConsumers - kBuilders, b, p0);
  }
  lds_barrier();  // results staged
  if constexpr (!NH) {
    // rows of 4 positions (8 bytes: H W is a multiple of 4) to y[b][o0 + row][p0 ..]
    constexpr int kQuads = L::MT / 4;
    for (int i = threadIdx.x; i < L::NE * kQuads; i += kThreads) {
      const int row = i / kQuads, c4 = i - row * kQuads;
      const int pos = p0 + 4 * c4, o = o0 + row;
      if (pos < p.HW && o < p.E) {
        const u32x2 val = *reinterpret_cast<const u32x2*>(smem + row * L::OROW + c4 * 8);
        __builtin_nontemporal_store(val, reinterpret_cast<u32x2*>(p.y + ((int64_t)b * p.E + o) * p.HW + pos));
      }
    }
    return;
  }
  // whole 16-byte pieces of the staged rows to y[b][p0 + row][o0 ..]
  constexpr int kPieces = L::NE / 8;
  for (int i = threadIdx.x; i < L::MT * kPieces; i += kThreads) {
    const int row = i / kPieces, c8 = i - row * kPieces;
    const int pos = p0 + row, o = o0 + 8 * c8;
    if (pos < p.HW && o < p.E) {
      const u32x4 val = *reinterpret_cast<const u32x4*>(smem + row * L::OROW + c8 * 16);
      __builtin_nontemporal_store(val, reinterpret_cast<u32x4*>(p.y + ((int64_t)b * p.HW + pos) * p.E + o));
    }
  }
}

using GmKernel = void (*)(GmArgs);

template <int MB, int NB, int NS, int OCC, bool NH>
size_t lds_of() { return Layout<MB, NB, NS, OCC, NH>::bytes(); }

struct Variant {
  int MB, NB, NS, OCC;
  bool NH;
  GmKernel k;
  size_t (*lds)();
};

constexpr int kParts = 2;

const Variant kVariants[] = {
    {4, 4, 2, 1, true, k_gmix<4, 4, 2, 1, true>, lds_of<4, 4, 2, 1, true>},
    {4, 3, 2, 1, true, k_gmix<4, 3, 2, 1, true>, lds_of<4, 3, 2, 1, true>},
    {7, 2, 2, 1, true, k_gmix<7, 2, 2, 1, true>, lds_of<7, 2, 2, 1, true>},
    {5, 3, 2, 1, true, k_gmix<5, 3, 2, 1, true>, lds_of<5, 3, 2, 1, true>},
    {4, 4, 2, 1, false, k_gmix<4, 4, 2, 1, false>, lds_of<4, 4, 2, 1, false>},
    {4, 3, 2, 1, false, k_gmix<4, 3, 2, 1, false>, lds_of<4, 3, 2, 1, false>},
    {7, 2, 2, 1, false, k_gmix<7, 2, 2, 1, false>, lds_of<7, 2, 2, 1, false>},
    {5, 3, 2, 1, false, k_gmix<5, 3, 2, 1, false>, lds_of<5, 3, 2, 1, false>},
};

int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  return cus;
}

// The variant with the least modelled time: rounds of workgroups over the
// CUs times the products one workgroup issues per step.
const Variant* pick(const Shape& sh) {
  const int64_t nblk = (sh.E + 15) / 16;
  const int cus = cu_count();
  const Variant* best = nullptr;
  int64_t best_cost = 0;
  for (const Variant& v : kVariants) {
    if (v.NS != kParts || v.NH != (sh.layout == MOCE_NHWC)) continue;
    if (v.lds() * v.OCC > (size_t)kLdsBytes) continue;
    const int64_t nt = (sh.HW + 16 * v.MB - 1) / (16 * v.MB);
    const int64_t nq = (nblk + 4 * v.NB - 1) / (4 * v.NB);
    const int64_t units = sh.B * nt * nq;
    const int64_t rounds = (units + cus - 1) / cus;
    const int64_t cost = rounds * v.MB * v.NB;
    if (!best || cost < best_cost || (cost == best_cost && v.NB > best->NB)) {
      best = &v;
      best_cost = cost;
    }
  }
  return best;
}

struct SchedShape {
  int nq, nbuckets, nsteps, cap;
  size_t off_bytes, total;
};

SchedShape sched_shape(const Shape& sh, const Variant& v) {
  SchedShape s{};
  const int nblk = (int)((sh.E + 15) / 16);
  s.nq = (nblk + 4 * v.NB - 1) / (4 * v.NB);
  s.nbuckets = s.nq * kBuilders;
  s.nsteps = (int)(sh.C / kStep);
  s.cap = kGroupsPerBuilder * kGroup * sh.k + (int)sh.C;
  s.off_bytes = ((size_t)s.nbuckets * (s.nsteps + 1) * 4 + 255) / 256 * 256;
  s.total = s.off_bytes + (size_t)s.nbuckets * s.cap * 8;
  return s;
}

}  // namespace

bool gmix_eligible(const Shape& sh) {
  if (sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.C % kStep != 0 || sh.C > kStep * kMaxSteps || sh.E % 8 != 0) return false;
  // channels-first rows start 8-byte aligned and are copied 4 bytes at a time
  if (sh.layout == MOCE_NCHW && sh.HW % 4 != 0) return false;
  if ((int64_t)sh.B * sh.HW > INT32_MAX / 2) return false;
  return pick(sh) != nullptr;
}

size_t gmix_sched_bytes(const Shape& sh) {
  const Variant* v = pick(sh);
  return v ? sched_shape(sh, *v).total : 0;
}

hipError_t launch_pool_sched(const Shape& sh, const void* x, float* d, const int32_t* s, const float* w,
                             const int32_t* U, int nU, void* sched, hipStream_t st) {
  const Variant* v = pick(sh);
  if (!v) return hipErrorInvalidValue;
  const SchedShape ss = sched_shape(sh, *v);
  SchedArgs a{};
  a.s = s;
  a.w = w;
  a.U = nU > 0 ? U : s;
  a.nU = nU;
  a.R = sh.R;
  a.k = sh.k;
  a.nsteps = ss.nsteps;
  a.cap = ss.cap;
  a.ng = 4 * v->NB;
  a.ngroups = (int)((sh.E + kGroup - 1) / kGroup);
  a.nbuckets = ss.nbuckets;
  a.off = static_cast<int32_t*>(sched);
  a.ent = reinterpret_cast<uint2*>(static_cast<char*>(sched) + ss.off_bytes);
  if (sh.layout == MOCE_NCHW && !(sh.HW % 8 == 0 && sh.HW / 8 >= 256)) {
    // channels-first planes pooled 8 bytes at a time, beside the schedule
    const int64_t planes = sh.B * sh.C;
    const int L = planes8_lanes(sh.HW);
    const int64_t per = kPoolThreads / L;
    const unsigned grid = (unsigned)(ss.nbuckets + std::min<int64_t>((planes + per - 1) / per, 32768));
    const uint16_t* xb = static_cast<const uint16_t*>(x);
    const int HW = (int)sh.HW;
    switch (L) {
      case 64: hipLaunchKernelGGL(k_pool_sched_planes<64>, dim3(grid), dim3(kPoolThreads), 0, st, xb, d, planes, HW, a); break;
      case 32: hipLaunchKernelGGL(k_pool_sched_planes<32>, dim3(grid), dim3(kPoolThreads), 0, st, xb, d, planes, HW, a); break;
      case 16: hipLaunchKernelGGL(k_pool_sched_planes<16>, dim3(grid), dim3(kPoolThreads), 0, st, xb, d, planes, HW, a); break;
      default: hipLaunchKernelGGL(k_pool_sched_planes<8>, dim3(grid), dim3(kPoolThreads), 0, st, xb, d, planes, HW, a); break;
    }
    return hipGetLastError();
  }
  if (sh.layout == MOCE_NCHW) {
    // long aligned planes: the plane pooling kernel, then the schedule alone
    const hipError_t e = launch_pool(sh, x, d, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_pool_sched<uint16_t>), dim3((unsigned)ss.nbuckets), dim3(kPoolThreads), 0, st,
                       static_cast<const uint16_t*>(x), d, (int)sh.C, (int)sh.HW, 1, a);
    return hipGetLastError();
  }
  const int nblk = (int)((sh.C / PoolVec<uint16_t>::EPV + 31) / 32);
  const unsigned grid = (unsigned)(ss.nbuckets + sh.B * nblk);
  hipLaunchKernelGGL((k_pool_sched<uint16_t>), dim3(grid), dim3(kPoolThreads), 0, st,
                     static_cast<const uint16_t*>(x), d, (int)sh.C, (int)sh.HW, nblk, a);
  return hipGetLastError();
}

hipError_t launch_gmix(const Shape& sh, const void* x, const float* stats, int nU, const void* sched, void* y,
                       hipStream_t st, const Epi& ep) {
  const Variant* v = pick(sh);
  if (!v) return hipErrorInvalidValue;
  const SchedShape ss = sched_shape(sh, *v);
  GmArgs p{};
  p.x = static_cast<const uint16_t*>(x);
  p.y = static_cast<uint16_t*>(y);
  p.off = static_cast<const int32_t*>(sched);
  p.ent = reinterpret_cast<const uint2*>(static_cast<const char*>(sched) + ss.off_bytes);
  p.st = stats;
  p.nst = sh.B * sh.R;
  p.C = (int)sh.C;
  p.HW = (int)sh.HW;
  p.E = sh.E;
  p.R = sh.R;
  p.nU = nU;
  p.nsteps = ss.nsteps;
  p.ngroups = (int)((sh.E + kGroup - 1) / kGroup);
  p.cap = ss.cap;
  p.nt = (int)((sh.HW + 16 * v->MB - 1) / (16 * v->MB));
  p.nq = ss.nq;
  p.units = (int)(sh.B * p.nt * p.nq);
  p.per = (p.units + 7) / 8;
  p.inv_nU = nU > 0 ? 1.f / (float)nU : 0.f;
  p.ep = ep;
  const size_t lds = v->lds();
  hipError_t e = hipFuncSetAttribute((const void*)v->k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(v->k, dim3(8 * p.per), dim3(threads_of(v->NH)), lds, st, p);
  return hipGetLastError();
}

}  // namespace moce

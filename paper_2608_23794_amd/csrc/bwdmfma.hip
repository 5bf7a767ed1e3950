// Matrix-core kernels of the backward.
//
// dalpha[b][e][i] = sum_p dy[b][e][p] x[b][s_ei][p] is a sampled product: for
// a block of Et experts and 256 channels it is the dense block
// G[e][c] = sum_p dy[b][e][p] x[b][c][p], of which only the support entries
// are kept.  With k/C small the dense block wastes most of its products, but
// the matrix cores run them at many times the rate of a gather through LDS
// (one LDS read per product), so the dense block is the faster way to the
// sparse result; both operands are the bfloat16 inputs themselves, exact in
// the products, accumulated in float32.
//
// A workgroup owns (expert block, channel block) and walks a set of units
// (image, range of positions).  Per unit, 32-position steps of both operands
// are staged in LDS (double-buffered, one barrier per step) and each of the
// 4 WE waves (WE = 1 or 2: at most two waves a SIMD, for the registers of
// the accumulators, operands and the loads in flight) accumulates a 64 x 64
// block as 4 x 4 MFMA 16x16x32 tiles.  A
// byte table [channel][expert] of support positions (0xff: not an entry),
// built once per workgroup from the prepared rows, picks the entries out of
// the accumulators at the end of a unit.
//
// Layouts in LDS:
//  - NCHW (positions contiguous): a row of 32 positions per feature (64
//    bytes), its four 16-byte chunks XOR-swizzled by (row >> 2) & 3, read as
//    one 16-byte operand per lane;
//  - channels-last: the 32 positions as rows of features (512 bytes for the
//    256 channels, at least 256 for the experts), 32-byte blocks
//    XOR-swizzled by the position, read as operands with the transposing LDS
//    load (two 8-byte loads per operand).
// Both swizzles make the operand reads and the staging writes free of bank
// conflicts.
#include <algorithm>
#include <climits>

#include "moce_internal.h"

namespace moce {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kDaWC = 4;       // channel waves: 4 x 64 = 256 channels per workgroup
constexpr int kDaCt = 64 * kDaWC;
constexpr int kDaKs = 32;      // positions per step
constexpr int kDaMaxK = 255;   // support positions fit a byte, 0xff marks "no entry"
constexpr int kDaTargetBlocks = 512;

// 32-byte block swizzle of the channels-last staging rows (16 blocks a row)
__device__ __forceinline__ int rowswz(int p) { return (p & 3) | ((p >> 1) & 4); }

template <int WE, bool NHWC, int VEC>
struct DaCfg {
  static constexpr int Et = 64 * WE;
  static constexpr int T = 64 * WE * kDaWC;
  // staging bytes of one step: A (experts) then B (channels)
  // channels-last rows: at least 256 bytes, so that the 8 values of the
  // block swizzle stay within the row
  static constexpr int APitch = NHWC ? (Et > 128 ? Et : 128) * 2 : 64;
  static constexpr int ABytes = NHWC ? kDaKs * APitch : Et * kDaKs * 2;
  static constexpr int BBytes = NHWC ? kDaKs * 256 * 2 : kDaCt * kDaKs * 2;
  static constexpr int Stage = ABytes + BBytes;
  static constexpr int TableBytes = kDaCt * Et;
  static constexpr int Lds = TableBytes + 2 * Stage;
  // 16-byte (NHWC) or VEC-position (NCHW) loads per step
  static constexpr int NA = NHWC ? kDaKs * Et / 8 : Et * (kDaKs / VEC);
  static constexpr int NB = NHWC ? kDaKs * kDaCt / 8 : kDaCt * (kDaKs / VEC);
  static constexpr int LPT = (NA + NB + T - 1) / T;
  static constexpr int WORDS = NHWC ? 4 : VEC / 2;  // 32-bit words per load
};

template <int WE, bool NHWC, int VEC>
__global__ void __launch_bounds__(64 * WE * kDaWC)
k_bwd_dalpha_mfma(const uint16_t* __restrict__ x, const uint16_t* __restrict__ dy, const int32_t* __restrict__ s,
                  float* __restrict__ dal, int B, int C, int E, int R, int k, int HW, int nsplit, int split_len,
                  int nCB, int G) {
  using Cf = DaCfg<WE, NHWC, VEC>;
  constexpr int Et = Cf::Et, T = Cf::T;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  unsigned char* table = lds;
  unsigned char* stage0 = lds + Cf::TableBytes;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int we = wave / kDaWC, wc = wave % kDaWC;
  const int g = blockIdx.x % G;
  const int rest = blockIdx.x / G;
  const int cb = rest % nCB, eb = rest / nCB;
  const int e0 = eb * Et, c0 = cb * kDaCt;

  // ---- the support-position table of this block: each wave takes 16 rows,
  // lanes along the row, all 16 loads of a chunk issued before any is used
  for (int q = tid; q < Cf::TableBytes / 16; q += T)
    reinterpret_cast<u32x4*>(table)[q] = u32x4{~0u, ~0u, ~0u, ~0u};
  __syncthreads();
  for (int i0 = 0; i0 < k; i0 += 64) {
    const int i = i0 + lane;
    int cv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int e = e0 + wave * 16 + r;
      cv[r] = s[(int64_t)min(e, R - 1) * k + min(i, k - 1)];
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int el = wave * 16 + r;
      const int cl = cv[r] - c0;
      if (e0 + el < R && i < k && cl >= 0 && cl < kDaCt)
        table[cl * Et + ((((el >> 2) ^ (cl & 15))) << 2) + (el & 3)] = (unsigned char)i;
    }
  }

  // ---- the units (image, position range) of this workgroup as one stream of
  // 32-position steps: the next step's loads are in flight while the current
  // one is multiplied, across unit boundaries too
  const int nunits = B * nsplit;
  auto unit_steps = [&](int u) {
    const int sp = u % nsplit;
    const int pb = sp * split_len, pe = min(HW, pb + split_len);
    return (pe - pb + kDaKs - 1) / kDaKs;
  };
  typedef uint32_t Regs[Cf::LPT][Cf::WORDS];
  // global -> registers for step ks of unit u (zeros outside the positions, experts and channels)
  auto load = [&](int u, int ks, Regs& reg) {
    const int b = u / nsplit, sp = u - b * nsplit;
    const int pb = sp * split_len, pe = min(HW, pb + split_len);
    const int p0 = pb + ks * kDaKs;
    const uint16_t* xb = x + (int64_t)b * C * HW;
    const uint16_t* yb = dy + (int64_t)b * E * HW;
#pragma unroll
    for (int j = 0; j < Cf::LPT; ++j) {
      const int q = tid + j * T;
#pragma unroll
      for (int w = 0; w < Cf::WORDS; ++w) reg[j][w] = 0;
      if (q < Cf::NA + Cf::NB) {
        const bool isA = q < Cf::NA;
        const int qq = isA ? q : q - Cf::NA;
        if (NHWC) {
          const int F = isA ? Et : kDaCt;
          const int p = qq / (F / 8), f8 = qq - p * (F / 8);
          const int f = (isA ? e0 : c0) + f8 * 8;
          const int nf = isA ? E : C;
          const int pp = p0 + p;
          if (pp < pe && f < nf) {
            const uint16_t* src = (isA ? yb : xb) + (int64_t)pp * nf + f;
            const u32x4 v = *reinterpret_cast<const u32x4*>(src);
            reg[j][0] = v.x;
            reg[j][1] = v.y;
            reg[j][2] = v.z;
            reg[j][3] = v.w;
          }
        } else {
          constexpr int CH = kDaKs / VEC;
          const int row = qq / CH, ch = qq - row * CH;
          const int f = (isA ? e0 : c0) + row;
          const int nf = isA ? E : C;
          const int pp = p0 + ch * VEC;
          if (pp < pe && f < nf) {
            const uint16_t* src = (isA ? yb : xb) + (int64_t)f * HW + pp;
            if (VEC == 8) {
              const u32x4 v = *reinterpret_cast<const u32x4*>(src);
              reg[j][0] = v.x;
              reg[j][1] = v.y;
              reg[j][2] = v.z;
              reg[j][3] = v.w;
            } else {
              const u32x2 v = *reinterpret_cast<const u32x2*>(src);
              reg[j][0] = v.x;
              reg[j][1] = v.y;
            }
          }
        }
      }
    }
  };
  // registers -> LDS stage buffer
  auto store = [&](unsigned char* stg, const Regs& reg) {
#pragma unroll
    for (int j = 0; j < Cf::LPT; ++j) {
      const int q = tid + j * T;
      if (q >= Cf::NA + Cf::NB) continue;
      const bool isA = q < Cf::NA;
      const int qq = isA ? q : q - Cf::NA;
      unsigned char* base = stg + (isA ? 0 : Cf::ABytes);
      if (NHWC) {
        const int F = isA ? Et : kDaCt;
        const int p = qq / (F / 8), f8 = qq - p * (F / 8);
        const int blk = (f8 >> 1) ^ rowswz(p);
        *reinterpret_cast<u32x4*>(base + p * (isA ? Cf::APitch : 512) + (blk << 5) + ((f8 & 1) << 4)) =
            u32x4{reg[j][0], reg[j][1], reg[j][2], reg[j][3]};
      } else {
        constexpr int CH = kDaKs / VEC;
        const int row = qq / CH, ch = qq - row * CH;
        // byte offset of positions ch*VEC.. within the row's 64 bytes
        const int off = ch * VEC * 2;
        const int chunk = (off >> 4) ^ ((row >> 2) & 3);
        unsigned char* dst = base + row * 64 + (chunk << 4) + (off & 15);
        if (VEC == 8)
          *reinterpret_cast<u32x4*>(dst) = u32x4{reg[j][0], reg[j][1], reg[j][2], reg[j][3]};
        else
          *reinterpret_cast<u32x2*>(dst) = u32x2{reg[j][0], reg[j][1]};
      }
    }
  };
  // operand of the 16-feature tile starting at feature fl of region `base`
  auto operand = [&](const unsigned char* base, int pitch, int fl) -> bf16x8 {
    if (NHWC) {
      const int G4 = lane >> 4, t = (lane >> 2) & 3, q = lane & 3;
      const int nb = fl >> 4;
      const int p1 = 8 * G4 + t, p2 = p1 + 4;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4*)(base + p1 * pitch + ((nb ^ rowswz(p1)) << 5) + (q << 3)));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4*)(base + p2 * pitch + ((nb ^ rowswz(p2)) << 5) + (q << 3)));
      typedef short s16x8 __attribute__((ext_vector_type(8)));
      const s16x8 v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      return __builtin_bit_cast(bf16x8, v);
    } else {
      const int row = fl + (lane & 15);
      const int chunk = (lane >> 4) ^ ((row >> 2) & 3);
      return *reinterpret_cast<const bf16x8*>(base + row * 64 + (chunk << 4));
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int me = 0; me < 4; ++me)
#pragma unroll
    for (int nc = 0; nc < 4; ++nc) acc[me][nc] = f32x4{0.f, 0.f, 0.f, 0.f};

  // steps as (unit, step within the unit); u >= nunits: past the end
  auto advance = [&](int& su, int& sk) {
    if (su >= nunits) return;
    if (++sk >= unit_steps(su)) {
      su += G;
      sk = 0;
    }
  };
  // step i is multiplied from LDS buffer i & 1 while step i + 1 waits in
  // registers (loaded an iteration earlier) and step i + 2 is being loaded
  Regs r0, r1;
  int u = g, ks = 0;             // step i
  int u1 = u, k1 = ks;           // step i + 1
  advance(u1, k1);
  int u2 = u1, k2 = k1;          // step i + 2
  advance(u2, k2);
  load(u, ks, r0);
  store(stage0, r0);
  if (u1 < nunits) load(u1, k1, r1);
  __syncthreads();  // the table and the first step
  int cur = 0;
  auto body = [&](Regs& rfree, Regs& rnext) {
    if (u2 < nunits) load(u2, k2, rfree);
    const unsigned char* stg = stage0 + cur * Cf::Stage;
    bf16x8 a[4], bb[4];
#pragma unroll
    for (int me = 0; me < 4; ++me) a[me] = operand(stg, Cf::APitch, 64 * we + 16 * me);
#pragma unroll
    for (int nc = 0; nc < 4; ++nc) bb[nc] = operand(stg + Cf::ABytes, 512, 64 * wc + 16 * nc);
#pragma unroll
    for (int me = 0; me < 4; ++me)
#pragma unroll
      for (int nc = 0; nc < 4; ++nc)
        acc[me][nc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[me], bb[nc], acc[me][nc], 0, 0, 0);
    if (ks + 1 == unit_steps(u)) {
      // ---- the support entries of unit u out of the accumulators
      const int b = u / nsplit, sp = u - b * nsplit;
      float* out = dal + (((int64_t)sp * B + b) * R) * k;
#pragma unroll
      for (int me = 0; me < 4; ++me)
#pragma unroll
        for (int nc = 0; nc < 4; ++nc) {
          const int cl = 64 * wc + 16 * nc + (lane & 15);
          const int el = 64 * we + 16 * me + 4 * (lane >> 4);
          const uint32_t word =
              *reinterpret_cast<const uint32_t*>(table + cl * Et + ((((el >> 2) ^ (cl & 15))) << 2));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const uint32_t pos = (word >> (8 * r)) & 0xffu;
            if (pos != 0xffu) out[(int64_t)(e0 + el + r) * k + pos] = acc[me][nc][r];
          }
          acc[me][nc] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }
    if (u1 < nunits) store(stage0 + (cur ^ 1) * Cf::Stage, rnext);
    __syncthreads();
    cur ^= 1;
    u = u1;
    ks = k1;
    u1 = u2;
    k1 = k2;
    advance(u2, k2);
  };
  while (u < nunits) {
    body(r0, r1);   // r0 held step i (already in LDS); step i + 1 sits in r1
    if (u >= nunits) break;
    body(r1, r0);
  }
}

template <int WE, bool NHWC, int VEC>
hipError_t launch_da(const Shape& sh, const uint16_t* x, const uint16_t* dy, const int32_t* s, float* dal,
                     int nsplit, int split_len, hipStream_t st) {
  using Cf = DaCfg<WE, NHWC, VEC>;
  const int nEB = (sh.R + Cf::Et - 1) / Cf::Et;
  const int nCB = (int)((sh.C + kDaCt - 1) / kDaCt);
  const int units = (int)sh.B * nsplit;
  int G = std::max(1, kDaTargetBlocks / (nEB * nCB));
  G = std::min(units, (G + 7) / 8 * 8);
  auto kern = k_bwd_dalpha_mfma<WE, NHWC, VEC>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, Cf::Lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(nEB * nCB * G), dim3(Cf::T), Cf::Lds, st, x, dy, s, dal, (int)sh.B, (int)sh.C,
                     sh.E, sh.R, sh.k, (int)sh.HW, nsplit, split_len, nCB, G);
  return hipGetLastError();
}

bool dalpha_mfma_eligible(const Shape& sh) {
  if (sh.elem != MOCE_BF16 || sh.R < 1 || sh.k > kDaMaxK) return false;
  if (sh.layout == MOCE_NHWC) return sh.C % 8 == 0 && sh.E % 8 == 0;
  return sh.HW % 4 == 0;
}

// Position splits of the NCHW product (units of work along the positions when
// the images alone give too few workgroups); dal then holds one partial sum
// per split.  1 wherever the matrix-core kernel does not apply.
void bwd_dalpha_split(const Shape& sh, int* nsplit, int* split_len) {
  *nsplit = 1;
  *split_len = (int)std::min<int64_t>(sh.HW, INT32_MAX / 2);
  if (!dalpha_mfma_eligible(sh) || sh.layout != MOCE_NCHW) return;
  const int WE = std::min(2, (sh.R + 63) / 64);
  const int64_t blocks = sh.B * ((sh.R + 64 * WE - 1) / (64 * WE)) * ((sh.C + kDaCt - 1) / kDaCt);
  const int64_t steps = (sh.HW + kDaKs - 1) / kDaKs;
  const int64_t want = std::min<int64_t>(steps, std::max<int64_t>(1, kDaTargetBlocks / std::max<int64_t>(1, blocks)));
  const int64_t len = (steps + want - 1) / want * kDaKs;
  *split_len = (int)len;
  *nsplit = (int)((sh.HW + len - 1) / len);
}

}  // namespace

void bwd_dalpha_splits(const Shape& sh, int* nsplit, int* split_len) { bwd_dalpha_split(sh, nsplit, split_len); }

bool bwd_mfma_dalpha(const Shape& sh, const void* x, const void* dy, const int32_t* s, const BwdWs& ws,
                     hipStream_t st, hipError_t* err) {
  if (!dalpha_mfma_eligible(sh)) return false;
  int nsplit, split_len;
  bwd_dalpha_split(sh, &nsplit, &split_len);
  const int WE = std::min(2, (sh.R + 63) / 64);
  auto xx = static_cast<const uint16_t*>(x);
  auto yy = static_cast<const uint16_t*>(dy);
#define MOCE_DA(W, N, V) launch_da<W, N, V>(sh, xx, yy, s, ws.dal, nsplit, split_len, st)
  if (sh.layout == MOCE_NHWC)
    *err = WE == 1 ? MOCE_DA(1, true, 8) : MOCE_DA(2, true, 8);
  else if (sh.HW % 8 == 0)
    *err = WE == 1 ? MOCE_DA(1, false, 8) : MOCE_DA(2, false, 8);
  else
    *err = WE == 1 ? MOCE_DA(1, false, 4) : MOCE_DA(2, false, 4);
#undef MOCE_DA
  return true;
}

// ---- dx on the matrix cores -------------------------------------------------
//
// dx[b][c][p] = sum_e coef_b[c][e] dy[b][e][p] + dd[b][c] / HW, where
// coef_b[c][e] is alpha_b[e][i] for the support entry (e, i) on channel c,
// 1/|U| for e = E-1 (the residual) when c is uncovered, and 0 elsewhere.
// The coefficients enter the product as two bf16 parts (hi = bf16(alpha),
// lo = bf16(alpha - hi): 16 significant bits), dy as it is.
//
// A per-call schedule sorts the entries (routed ones and one residual entry
// per uncovered channel) into buckets by (block of 256 channels, chunk of 64
// experts); a second pass writes, per image and in schedule order, each
// entry's two coefficient parts packed in 32 bits.  A workgroup owns (image,
// 64 positions, 256 channels) and walks the expert chunks: the chunk's dy
// tile (64 x 64) and its coefficient tile (256 x 64, two parts) sit in LDS,
// double-buffered; the coefficient tile starts zero, receives its bucket's
// entries by scatter and is cleared entry by entry once multiplied, so a
// chunk costs LDS writes in proportion to its entries, not to its area.
// The bucket entries are prefetched two chunks ahead and a chunk's scatter
// into the idle buffer runs beside the products of the current chunk.
namespace {

constexpr int kDxCt = 256;   // channels per workgroup
constexpr int kDxEk = 64;    // experts per chunk
constexpr int kDxP = 64;     // positions per workgroup
constexpr int kDxThreads = 512;
constexpr int kDxEPT = 4;    // bucket entries a thread holds for the next scatter
constexpr int kDxCoefPart = kDxCt * kDxEk * 2;   // bytes of one part of one buffer
constexpr int kDxCoefBuf = 2 * kDxCoefPart;
constexpr int kDxDyBuf = kDxP * kDxEk * 2;
constexpr int kDxLds = 2 * kDxCoefBuf + 2 * kDxDyBuf;

__global__ void k_dxs_fill(int32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// the bucket of entry t: routed t < R k (channel s[t], expert t / k), else the
// residual entry of channel t - R k when that channel has no routed entry
__device__ __forceinline__ bool dxs_entry(int64_t t, const int32_t* s, const int32_t* cnt, int R, int k, int nEC,
                                          int* key, int* c, int* e) {
  const int64_t rk = (int64_t)R * k;
  if (t < rk) {
    *c = s[t];
    *e = (int)(t / k);
  } else {
    *c = (int)(t - rk);
    if (cnt[*c] != 0) return false;
    *e = R;
  }
  *key = (*c / kDxCt) * nEC + *e / kDxEk;
  return true;
}

// Bucket counts, aggregated per workgroup in LDS (one global atomic per
// bucket and workgroup): kDxEntPerBlock entries per workgroup.
constexpr int kDxEntPerBlock = 4096;
constexpr int kDxMaxBuckets = 4096;

__global__ void __launch_bounds__(256)
k_dxs_count(const int32_t* __restrict__ s, const int32_t* __restrict__ cnt, int R, int k, int C, int nEC, int nb,
            int32_t* __restrict__ bcnt) {
  __shared__ int32_t local[kDxMaxBuckets];
  for (int i = threadIdx.x; i < nb; i += 256) local[i] = 0;
  __syncthreads();
  const int64_t n = (int64_t)R * k + C;
  const int64_t t0 = (int64_t)blockIdx.x * kDxEntPerBlock;
  for (int j = threadIdx.x; j < kDxEntPerBlock; j += 256) {
    const int64_t t = t0 + j;
    int key, c, e;
    if (t < n && dxs_entry(t, s, cnt, R, k, nEC, &key, &c, &e)) atomicAdd(&local[key], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nb; i += 256)
    if (local[i]) atomicAdd(&bcnt[i], local[i]);
}

// one thread: exclusive scan of the bucket counts into boff[0..nb], bcur = boff
__global__ void k_dxs_scan(const int32_t* __restrict__ bcnt, int nb, int32_t* __restrict__ boff,
                           int32_t* __restrict__ bcur) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  int32_t run = 0;
  for (int i = 0; i < nb; ++i) {
    boff[i] = run;
    bcur[i] = run;
    run += bcnt[i];
  }
  boff[nb] = run;
}

// w0 = channel within the block | expert within the chunk << 8; w1 = entry
// (e k + i) or -1 (residual).  Each workgroup reserves one range per bucket
// and places its entries inside it (the order within a bucket is free: every
// entry has its own place in the coefficient tile).
__global__ void __launch_bounds__(256)
k_dxs_place(const int32_t* __restrict__ s, const int32_t* __restrict__ cnt, int R, int k, int C, int nEC, int nb,
            int32_t* __restrict__ bcur, uint32_t* __restrict__ w0, int32_t* __restrict__ w1) {
  __shared__ int32_t local[kDxMaxBuckets];
  for (int i = threadIdx.x; i < nb; i += 256) local[i] = 0;
  __syncthreads();
  const int64_t n = (int64_t)R * k + C;
  const int64_t t0 = (int64_t)blockIdx.x * kDxEntPerBlock;
  for (int j = threadIdx.x; j < kDxEntPerBlock; j += 256) {
    const int64_t t = t0 + j;
    int key, c, e;
    if (t < n && dxs_entry(t, s, cnt, R, k, nEC, &key, &c, &e)) atomicAdd(&local[key], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nb; i += 256) local[i] = local[i] ? atomicAdd(&bcur[i], local[i]) : 0;
  __syncthreads();
  for (int j = threadIdx.x; j < kDxEntPerBlock; j += 256) {
    const int64_t t = t0 + j;
    int key, c, e;
    if (t < n && dxs_entry(t, s, cnt, R, k, nEC, &key, &c, &e)) {
      const int pos = atomicAdd(&local[key], 1);
      w0[pos] = (uint32_t)(c % kDxCt) | ((uint32_t)(e % kDxEk) << 8);
      w1[pos] = t < (int64_t)R * k ? (int32_t)t : -1;
    }
  }
}

// the two bf16 parts of each scheduled entry's coefficient, per image
__global__ void k_dxs_alpha(const int32_t* __restrict__ w1, const int32_t* __restrict__ boff, int nb,
                            const float* __restrict__ w, const float* __restrict__ stats,
                            const int32_t* __restrict__ nUp, int64_t B, int R, int k, int64_t NEmax,
                            uint32_t* __restrict__ coef) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t b = blockIdx.y;
  if (j >= boff[nb]) return;
  const int ent = w1[j];
  float a;
  if (ent >= 0) {
    const int e = ent / k;
    const int64_t row = b * R + e, n = B * R;
    a = coef_alpha(coef_e(coef_z(w[ent], stats[row]), stats[n + row]), stats[2 * n + row]);
  } else {
    a = 1.f / (float)*nUp;
  }
  const uint16_t hi = f32_to_bf16(a);
  const uint16_t lo = f32_to_bf16(a - bf16_to_f32(hi));
  coef[b * NEmax + j] = (uint32_t)hi | ((uint32_t)lo << 16);
}

__device__ __forceinline__ int dyswz(int r) { return ((r >> 1) & 1) | ((r >> 2) & 2); }

// byte offset of (channel cl, expert el) in one coefficient part: rows of 64
// experts (128 bytes), 16-byte chunks XOR-swizzled by the channel
__device__ __forceinline__ int coef_off(int cl, int el) {
  return cl * 128 + ((((el >> 3) ^ (cl & 7))) << 4) + ((el & 7) << 1);
}

template <bool NHWC, int VEC>
__global__ void __launch_bounds__(kDxThreads)
k_bwd_dx_mfma(const uint16_t* __restrict__ dy, uint16_t* __restrict__ dx, const float* __restrict__ dd,
              const int32_t* __restrict__ boff, const uint32_t* __restrict__ w0, const uint32_t* __restrict__ coefs,
              int B, int C, int E, int HW, int nEC, int nCB, int nPC, int64_t NEmax) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  unsigned char* coefL = lds;                         // [2 buf][2 part][256][64] bf16
  unsigned char* dyL = lds + 2 * kDxCoefBuf;          // [2 buf][64][64] bf16
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t units = (int64_t)B * nPC;
  const int cb = (int)(blockIdx.x / units);
  const int64_t bp = blockIdx.x - (int64_t)cb * units;
  const int b = (int)(bp / nPC), pc = (int)(bp - (int64_t)b * nPC);
  const int c0 = cb * kDxCt, p0 = pc * kDxP;
  const uint16_t* yb = dy + (int64_t)b * E * HW;
  const uint32_t* cb_coef = coefs + (int64_t)b * NEmax;

  // zero both coefficient buffers once; every scatter is undone after use
  for (int q = tid; q < 2 * kDxCoefBuf / 16; q += kDxThreads)
    reinterpret_cast<u32x4*>(coefL)[q] = u32x4{0u, 0u, 0u, 0u};

  // a bucket's entries: the first kDxEPT * kDxThreads in registers, the rest
  // read again where they are used
  struct Ents {
    uint32_t w0[kDxEPT], cf[kDxEPT];
    int n, base;
  };
  auto load_entries = [&](int ec, Ents& E) {
    const int key = cb * nEC + ec;
    E.base = boff[key];
    E.n = boff[key + 1] - E.base;
#pragma unroll
    for (int r = 0; r < kDxEPT; ++r) {
      const int j = E.base + min(tid + r * kDxThreads, max(E.n - 1, 0));
      E.w0[r] = w0[j];
      E.cf[r] = cb_coef[j];
    }
  };
  // scatter (or, with clear, zero) a bucket's entries into buffer `buf`
  auto scatter = [&](int buf, const Ents& E, bool clear) {
    unsigned char* hiP = coefL + buf * kDxCoefBuf;
    unsigned char* loP = hiP + kDxCoefPart;
#pragma unroll
    for (int r = 0; r < kDxEPT; ++r) {
      if (tid + r * kDxThreads < E.n) {
        const int o = coef_off(E.w0[r] & 255, E.w0[r] >> 8);
        *reinterpret_cast<uint16_t*>(hiP + o) = clear ? 0 : (uint16_t)(E.cf[r] & 0xffff);
        *reinterpret_cast<uint16_t*>(loP + o) = clear ? 0 : (uint16_t)(E.cf[r] >> 16);
      }
    }
    for (int q = tid + kDxEPT * kDxThreads; q < E.n; q += kDxThreads) {
      const uint32_t v0 = w0[E.base + q], v1 = cb_coef[E.base + q];
      const int o = coef_off(v0 & 255, v0 >> 8);
      *reinterpret_cast<uint16_t*>(hiP + o) = clear ? 0 : (uint16_t)(v1 & 0xffff);
      *reinterpret_cast<uint16_t*>(loP + o) = clear ? 0 : (uint16_t)(v1 >> 16);
    }
  };
  // dy tile of expert chunk ec: NHWC rows of positions (64 experts each, 16-byte
  // chunks swizzled by the row), NCHW rows of experts (64 positions each,
  // 32-byte blocks swizzled for the transposing read)
  constexpr int DYL = NHWC ? 1 : 8 / VEC;   // loads per thread
  constexpr int DYW = NHWC ? 4 : VEC / 2;   // words per load
  uint32_t dyr[DYL][DYW];
  auto load_dy = [&](int ec) {
    const int e0 = ec * kDxEk;
#pragma unroll
    for (int j = 0; j < DYL; ++j) {
#pragma unroll
      for (int w = 0; w < DYW; ++w) dyr[j][w] = 0;
      if (NHWC) {
        const int row = tid >> 3, oct = tid & 7;
        const int p = p0 + row, e = e0 + oct * 8;
        if (p < HW && e < E) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(yb + (int64_t)p * E + e);
          dyr[j][0] = v.x;
          dyr[j][1] = v.y;
          dyr[j][2] = v.z;
          dyr[j][3] = v.w;
        }
      } else {
        const int q = tid + j * kDxThreads;
        constexpr int PER = kDxP / VEC;     // loads per expert row
        const int row = q / PER, piece = q - row * PER;
        const int e = e0 + row, p = p0 + piece * VEC;
        if (e < E && p < HW) {
          const uint16_t* src = yb + (int64_t)e * HW + p;
          if (VEC == 8) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(src);
            dyr[j][0] = v.x;
            dyr[j][1] = v.y;
            dyr[j][2] = v.z;
            dyr[j][3] = v.w;
          } else {
            const u32x2 v = *reinterpret_cast<const u32x2*>(src);
            dyr[j][0] = v.x;
            dyr[j][1] = v.y;
          }
        }
      }
    }
  };
  auto store_dy = [&](int buf) {
    unsigned char* base = dyL + buf * kDxDyBuf;
#pragma unroll
    for (int j = 0; j < DYL; ++j) {
      if (NHWC) {
        const int row = tid >> 3, oct = tid & 7;
        *reinterpret_cast<u32x4*>(base + row * 128 + ((oct ^ (row & 7)) << 4)) =
            u32x4{dyr[j][0], dyr[j][1], dyr[j][2], dyr[j][3]};
      } else {
        const int q = tid + j * kDxThreads;
        constexpr int PER = kDxP / VEC;
        const int row = q / PER, piece = q - row * PER;
        const int byte = piece * VEC * 2;               // within the 128-byte row
        const int blk = (byte >> 5) ^ dyswz(row);
        unsigned char* dst = base + row * 128 + (blk << 5) + (byte & 31);
        if (VEC == 8)
          *reinterpret_cast<u32x4*>(dst) = u32x4{dyr[j][0], dyr[j][1], dyr[j][2], dyr[j][3]};
        else
          *reinterpret_cast<u32x2*>(dst) = u32x2{dyr[j][0], dyr[j][1]};
      }
    }
  };

  f32x4 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  Ents E0, E1, E2;   // the entries of chunks ec, ec + 1, ec + 2
  load_entries(0, E0);
  load_dy(0);
  __syncthreads();  // the zeroed buffers
  scatter(0, E0, false);
  store_dy(0);
  if (nEC > 1) {
    load_entries(1, E1);
    load_dy(1);
  }
  __syncthreads();
  for (int ec = 0; ec < nEC; ++ec) {
    const int cur = ec & 1;
    if (ec + 1 < nEC) {   // chunk ec + 1 into the idle buffers, beside the products of chunk ec
      scatter(cur ^ 1, E1, false);
      store_dy(cur ^ 1);
    }
    if (ec + 2 < nEC) {
      load_entries(ec + 2, E2);
      load_dy(ec + 2);
    }
    const unsigned char* hiP = coefL + cur * kDxCoefBuf;
    const unsigned char* loP = hiP + kDxCoefPart;
    const unsigned char* dyP = dyL + cur * kDxDyBuf;
#pragma unroll
    for (int ks = 0; ks < kDxEk / 32; ++ks) {
      const int oct = ks * 4 + (lane >> 4);
      if (NHWC) {
        // D[p][c]: A = dy rows (positions), B = coefficient rows (channels)
        bf16x8 a[4], bh[2], bl[2];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          const int row = mt * 16 + (lane & 15);
          a[mt] = *reinterpret_cast<const bf16x8*>(dyP + row * 128 + ((oct ^ (row & 7)) << 4));
        }
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int cl = (wave * 2 + nt) * 16 + (lane & 15);
          const int o = cl * 128 + ((oct ^ (cl & 7)) << 4);
          bh[nt] = *reinterpret_cast<const bf16x8*>(hiP + o);
          bl[nt] = *reinterpret_cast<const bf16x8*>(loP + o);
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bh[nt], acc[mt][nt], 0, 0, 0);
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], bl[nt], acc[mt][nt], 0, 0, 0);
          }
      } else {
        // D[c][p]: A = coefficient rows (channels), B = dy rows (experts) read transposed
        bf16x8 ah[2], al[2], bb[4];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const int cl = (wave * 2 + mt) * 16 + (lane & 15);
          const int o = cl * 128 + ((oct ^ (cl & 7)) << 4);
          ah[mt] = *reinterpret_cast<const bf16x8*>(hiP + o);
          al[mt] = *reinterpret_cast<const bf16x8*>(loP + o);
        }
        const int G4 = lane >> 4, t = (lane >> 2) & 3, q = lane & 3;
        const int r1 = ks * 32 + 8 * G4 + t, r2 = r1 + 4;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_s16x4*)(dyP + r1 * 128 + ((nt ^ dyswz(r1)) << 5) + (q << 3)));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_s16x4*)(dyP + r2 * 128 + ((nt ^ dyswz(r2)) << 5) + (q << 3)));
          typedef short s16x8 __attribute__((ext_vector_type(8)));
          const s16x8 v = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          bb[nt] = __builtin_bit_cast(bf16x8, v);
        }
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[mt], bb[nt], acc[nt][mt], 0, 0, 0);
            acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[mt], bb[nt], acc[nt][mt], 0, 0, 0);
          }
      }
    }
    __syncthreads();  // every wave is done with buffer cur; chunk ec + 1 is in place
    scatter(cur, E0, true);
    __syncthreads();  // buffer cur is zero again before chunk ec + 2 goes in
    E0 = E1;
    E1 = E2;
  }

  // ---- epilogue: + dd / HW, rounded to bf16
  const float rhw = 1.f / (float)HW;
  if (NHWC) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int c = c0 + (wave * 2 + nt) * 16 + (lane & 15);
        if (c >= C) continue;
        const float add = dd[(int64_t)b * C + c] * rhw;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int p = p0 + mt * 16 + 4 * (lane >> 4) + r;
          if (p < HW) dx[((int64_t)b * HW + p) * C + c] = f32_to_bf16(acc[mt][nt][r] + add);
        }
      }
  } else {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = c0 + (wave * 2 + mt) * 16 + 4 * (lane >> 4) + r;
        if (c >= C) continue;
        const float add = dd[(int64_t)b * C + c] * rhw;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const int p = p0 + nt * 16 + (lane & 15);
          if (p < HW) dx[((int64_t)b * C + c) * HW + p] = f32_to_bf16(acc[nt][mt][r] + add);
        }
      }
  }
}

bool dx_mfma_eligible(const Shape& sh) {
  if (sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if ((sh.C + kDxCt - 1) / kDxCt * ((sh.E + kDxEk - 1) / kDxEk) > kDxMaxBuckets) return false;
  if (sh.layout == MOCE_NHWC) return sh.E % 8 == 0;
  return sh.HW % 4 == 0;
}

}  // namespace

void bwd_dx_sched_sizes(const Shape& sh, int* nbuckets, int64_t* ne_max) {
  const int nEC = (sh.E + kDxEk - 1) / kDxEk;
  const int nCB = (int)((sh.C + kDxCt - 1) / kDxCt);
  *nbuckets = dx_mfma_eligible(sh) ? nEC * nCB : 0;
  *ne_max = dx_mfma_eligible(sh) ? (int64_t)sh.R * sh.k + sh.C : 0;
}

bool bwd_mfma_dx(const Shape& sh, const void* dy, const int32_t* s, const float* w, const BwdWs& ws, void* dx,
                 hipStream_t st, hipError_t* err) {
  if (!dx_mfma_eligible(sh)) return false;
  int nb;
  int64_t NEmax;
  bwd_dx_sched_sizes(sh, &nb, &NEmax);
  const int nECb = (sh.E + kDxEk - 1) / kDxEk;
  const int nCB = (int)((sh.C + kDxCt - 1) / kDxCt);
  k_dxs_fill<<<(nb + 255) / 256, 256, 0, st>>>(ws.dxs_cnt, nb);
  const int64_t nt = NEmax;
  const unsigned gb = (unsigned)((nt + kDxEntPerBlock - 1) / kDxEntPerBlock);
  k_dxs_count<<<gb, 256, 0, st>>>(s, ws.cnt, sh.R, sh.k, (int)sh.C, nECb, nb, ws.dxs_cnt);
  k_dxs_scan<<<1, 64, 0, st>>>(ws.dxs_cnt, nb, ws.dxs_off, ws.dxs_cur);
  k_dxs_place<<<gb, 256, 0, st>>>(s, ws.cnt, sh.R, sh.k, (int)sh.C, nECb, nb, ws.dxs_cur, ws.dxs_w0, ws.dxs_w1);
  k_dxs_alpha<<<dim3((unsigned)((NEmax + 255) / 256), (unsigned)sh.B), 256, 0, st>>>(
      ws.dxs_w1, ws.dxs_off, nb, w, ws.stats, ws.nU, sh.B, sh.R, sh.k, NEmax, ws.dxs_coef);
  if ((*err = hipGetLastError()) != hipSuccess) return true;
  const int nPC = (int)((sh.HW + kDxP - 1) / kDxP);
  const unsigned grid = (unsigned)(nCB * sh.B * nPC);
  auto y = static_cast<const uint16_t*>(dy);
  auto o = static_cast<uint16_t*>(dx);
  using K = void (*)(const uint16_t*, uint16_t*, const float*, const int32_t*, const uint32_t*, const uint32_t*, int,
                     int, int, int, int, int, int, int64_t);
  const K kern = sh.layout == MOCE_NHWC ? k_bwd_dx_mfma<true, 8>
                 : sh.HW % 8 == 0      ? k_bwd_dx_mfma<false, 8>
                                       : k_bwd_dx_mfma<false, 4>;
  if ((*err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kDxLds)) !=
      hipSuccess)
    return true;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kDxThreads), kDxLds, st, y, o, ws.dd, ws.dxs_off, ws.dxs_w0,
                     ws.dxs_coef, (int)sh.B, (int)sh.C, sh.E, (int)sh.HW, nECb, nCB, nPC, NEmax);
  *err = hipGetLastError();
  return true;
}

}  // namespace moce

// Fused forward for NCHW bfloat16 inputs in a single pass over x: pooling
// (Sec. 3.2), temperatures and coefficients (Eqs. 3-4), routed experts
// (Eq. 5) and the residual output (Eq. 6) in one launch.
//
// Tiles.  Image b is cut into nt = ceil(HW / 64) tiles of 64 positions by
// all C (<= 256) channels; tile n of the batch is (b, j) = (n / nt, n % nt).
// A 512-thread workgroup keeps one tile in LDS, widened to float32, from the
// moment it is staged until it has been mixed, so x is read from HBM once:
// the per-channel sums that pooling needs are taken from the tile data on its
// way in.  Two workgroups share a CU, so that one computes while the other
// waits for memory or for a gate.
//
// Schedule.  The launch is cooperative: G mixing workgroups (two per CU,
// less the gate service below) are resident together, and mixing workgroup g
// takes tiles g, g + G, g + 2G, ...  At the step that mixes tile n, the data
// of tile n + G is already in registers and its channel sums are published
// first, then the loads of tile n + 2G are issued, so an image's channel sums
// are complete about one step before its tiles are mixed.
//
// Gate service.  The temperatures of image b depend on the mean of every
// channel over all of b's tiles.  The last NG (<= 16, two per XCD) workgroups
// of the launch do no mixing: each takes every NG-th image in order, polls its
// nt published channel sums of every channel, adds them in tile order (so
// the result does not depend on timing), and evaluates tau =
// softplus(a_o . d_S + c_o) + 1e-3 and the log-partition of softmax(w_o / tau)
// for every expert, a group of lanes per expert with the sums and maxima over
// its support entries taken by lane shuffles, the gate tables in registers.
// A gate is thus published about one memory round trip after the image's
// last channel sums, well before the image's tiles are mixed; the mixing
// workgroups only poll for the 2R values.
//
// Mixing.  Each quarter wave computes one expert and each lane 4 consecutive
// positions of the tile: a support entry costs one 16-byte LDS read and four
// FMAs.  The byte offsets of an expert's support rows are 16-bit values in
// LDS, read eight at a time, and the coefficients four at a time.
//
// Hand-off without fences.  Channel sums, temperatures and log-partitions
// start as a sentinel NaN (written by the fill kernel) and are published with
// system-scope stores; consumers poll them with system-scope loads.  Each
// value is its own ready flag, so no ordering between locations and no
// acquire or release fence is needed.
//
// Progress.  The gate service waits only for channel sums, which every mixing
// workgroup publishes for tile m at the start of the step that mixes m - G,
// before any wait of that step.  A mixing workgroup waits for the gate of
// image b while holding the unpublished tile n + 2G, which belongs to a later
// image because G >= nt; the workgroup of any tile m of b reaches the step that
// publishes m after mixing m - 2G, which belongs to an earlier image.  The
// service handles images in increasing order.  By induction over images every
// wait ends, given that all workgroups run at once, which the cooperative
// launch guarantees.  Every wait is in addition bounded (kSpinLimit polls); one
// that runs out sets err[0] and the kernel still terminates.
#include <algorithm>
#include <atomic>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr uint32_t kSentinel = 0x7FC0DEADu;
constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kTT = 64;              // positions per tile
constexpr int kRowBytes = kTT * 4;   // bytes of one channel row of the LDS tile
constexpr int kPerCU = 2;            // workgroups per CU
constexpr int kSpinLimit = 1 << 22;
constexpr int kMaxDevices = 64;
constexpr int kMaxLds = 80 * 1024 - 1024;  // per workgroup, leaving room for the static variables
constexpr int kWSlots = 4;                 // logits per thread held in registers
constexpr int kQuads = 8;                  // groups of four channel sums polled together
constexpr int kGateWorkgroups = 16;        // gate service workgroups (at most one per image)

struct FusedArgs {
  int B, C, HW, E, R, k, kq, nU;  // kq: k rounded up to a multiple of 8
  int nt, ntiles;                 // tiles per image, tiles in the batch
  int ntp;                        // nt rounded up to a multiple of 4: row length of the channel sums
  int gsz, epl;                   // gate lanes per expert (a power of two, 8 to 64), entries per lane
  int ng;                         // gate service workgroups (the last ng of the grid)
  int gated;                      // tau and lse are final on entry: no channel sums, no gate service
};

// LDS regions, in bytes: the tile [C][kTT] float; the coefficients [R][kq]
// float, also the gate's scratch (kThreads + C floats); the support row
// offsets [R][kq] uint16; the coefficient exponent factors [R] float2.
struct LdsLayout {
  size_t alpha, sofs, tl, total;
};

__host__ __device__ inline LdsLayout lds_layout(int C, int R, int kq) {
  LdsLayout l;
  l.alpha = (size_t)C * kTT * 4;
  const size_t alpha_floats = std::max((size_t)R * kq, (size_t)kThreads + C);
  l.sofs = l.alpha + alpha_floats * 4;
  l.tl = l.sofs + (((size_t)R * kq * 2 + 15) & ~(size_t)15);
  l.total = l.tl + (size_t)R * 8;
  return l;
}

__device__ __forceinline__ void publish(float* p, float v) {
  uint32_t u = __float_as_uint(v);
  if (u == kSentinel) u = 0x7FC00000u;  // never publish the sentinel itself
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// One relaxed system-scope load of a published value (may still be the sentinel).
__device__ __forceinline__ uint32_t peek_value(const float* p) {
  return __hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Polls p until it holds a published value (bounded; a timeout sets err[0]).
__device__ __forceinline__ float await_value(const float* p, int* err) {
  uint32_t u = peek_value(p);
  for (int n = 0; u == kSentinel && n < kSpinLimit; ++n) {
    __builtin_amdgcn_s_sleep(2);
    u = peek_value(p);
  }
  if (u == kSentinel) atomicOr(err, 1);
  return __uint_as_float(u);
}

// A value read earlier with peek_value, polled again only if it was not yet published.
__device__ __forceinline__ float settle_value(uint32_t peeked, const float* p, int* err) {
  return peeked != kSentinel ? __uint_as_float(peeked) : await_value(p, err);
}

__device__ __forceinline__ float sum8_bf16(uint4 v) {
  return ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
         ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
}

template <int Ctrl>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), Ctrl, 0xF, 0xF, false));
}

// Sum over each group of 8 lanes: lane pairs, quads, then the two quads of
// the group (row_half_mirror), with every lane receiving its group's total.
__device__ __forceinline__ float group8_sum(float v) {
  v += dpp_move<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_move<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_move<0x141>(v);  // row_half_mirror
  return v;
}

// Sum and maximum over aligned groups of gsz lanes (gsz a power of two, 8 to
// 64): DPP steps within rows of 16 lanes (pairs, quads, half rows, rows),
// then lane shuffles across rows, every lane receiving its group's result.
template <bool Max>
__device__ __forceinline__ float group_reduce(float v, int gsz) {
  auto op = [](float a, float b) { return Max ? fmaxf(a, b) : a + b; };
  v = op(v, dpp_move<0xB1>(v));   // quad_perm [1,0,3,2]
  v = op(v, dpp_move<0x4E>(v));   // quad_perm [2,3,0,1]
  v = op(v, dpp_move<0x141>(v));  // row_half_mirror
  if (gsz == 8) return v;
  v = op(v, dpp_move<0x140>(v));  // row_mirror
  if (gsz == 16) return v;
  v = op(v, __shfl_xor(v, 16, 64));
  if (gsz == 32) return v;
  return op(v, __shfl_xor(v, 32, 64));
}
__device__ __forceinline__ float group_sum(float v, int gsz) { return group_reduce<false>(v, gsz); }
__device__ __forceinline__ float group_max(float v, int gsz) { return group_reduce<true>(v, gsz); }

// Issues the global loads of tile n into buf (4 x 16 bytes per thread): thread
// t reads 8 positions of channel (t >> 3) + 64u in round u.  Lanes past the
// data load a clamped, in-bounds address; their data is masked where it is
// used (tile_valid), not here, so that nothing waits for the loads before
// the data is needed.
__device__ __forceinline__ void issue_tile(const FusedArgs& p, const uint16_t* __restrict__ x, int n, uint4* buf) {
  const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
  const int p0 = j * kTT;
  const int vvalid = min(kTT, p.HW - p0) / 8;
  const uint16_t* xb = x + (int64_t)b * p.C * p.HW + p0;
  const int qv = threadIdx.x & 7;
  // all four rounds load (rows past C repeat row C - 1), so that the loads
  // are straight-line code and the compiler's wait counting stays exact
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = (threadIdx.x >> 3) + u * 64;
    buf[u] = *reinterpret_cast<const uint4*>(xb + (int64_t)min(c, p.C - 1) * p.HW + min(qv, vvalid - 1) * 8);
  }
}

// Whether round u of this thread's loads of tile n holds real data.
__device__ __forceinline__ bool tile_valid(const FusedArgs& p, int n, int u) {
  const int j = n - (n / p.nt) * p.nt;
  const int vvalid = min(kTT, p.HW - j * kTT) / 8;
  return (int)(threadIdx.x >> 3) + u * 64 < p.C && (int)(threadIdx.x & 7) < vvalid;
}

// Gate service: workgroup gs of the last NG of the launch evaluates the gate
// of images gs, gs + NG, ... in that order.  For each image it polls the nt
// published channel sums of every channel, adds them in tile order (so the
// result does not depend on timing), and evaluates per expert (a group of gsz
// lanes, each lane epl support entries) g = c_o + sum_i a_o,i d[s_o,i],
// tau = softplus(g) + 1e-3 and the log-partition m + log(sum_i exp(w_o,i /
// tau - m)), publishing tau and the log-partition.  The gate tables of the
// first kGatePass passes stay in registers.  scratch holds kThreads + C floats.
constexpr int kGatePass = 4;

__device__ __forceinline__ void gate_service(const FusedArgs& p, int gs, int ng, const float* part, float* tau,
                                             float* lse, const int* arrive, int* err, const int32_t* __restrict__ s,
                                             const float* __restrict__ w, const float* __restrict__ ga,
                                             const float* __restrict__ gc, float* scratch) {
  float* red = scratch;             // [kThreads]
  float* dl = scratch + kThreads;   // [C]
  const int gpp = kThreads / p.gsz;  // experts per pass
  const int gl = threadIdx.x % p.gsz;
  const int npass = (p.R + gpp - 1) / gpp;
  const bool one = p.epl == 1;       // one support entry per lane

  float pa[kGatePass], pw[kGatePass], pc[kGatePass];
  int ps[kGatePass];
#pragma unroll
  for (int q = 0; q < kGatePass; ++q) {
    const int o = min(threadIdx.x / p.gsz + q * gpp, p.R - 1);
    const int64_t src = min((int64_t)o * p.k + gl, (int64_t)p.R * p.k - 1);
    pa[q] = ga[src];
    pw[q] = w[src];
    ps[q] = s[src];
    pc[q] = gc[o];
  }

  // thread t adds up the tiles of channel c = t % C in groups of four: groups
  // g = r, r + nsplit, ... with r = t / C, read as 16-byte system-scope
  // buffer loads (one scalar resource, 32-bit lane offsets); a batch that
  // meets a value not yet published is read again after a pause, until every
  // value of the batch is in
  const int nsplit = kThreads / p.C;
  const int c = threadIdx.x % p.C, r = threadIdx.x / p.C;
  const int nq = p.ntp / 4;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(part), 0, p.B * p.C * p.ntp * 4, 0x00020000);
  constexpr int kSysCoherent = 1 | 16;  // sc0 sc1
  __shared__ int sh_count;
  for (int b = gs; b < p.B; b += ng) {
    // wait (one lane, one word) until every tile of the image has counted
    // itself; the sums are read only then
    if (threadIdx.x == 0) {
      int n = 0, tries = 0;
      for (;;) {
        n = __hip_atomic_load(arrive + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        if (n >= p.nt || ++tries >= kSpinLimit) break;
        __builtin_amdgcn_s_sleep(8);
      }
      sh_count = n;
    }
    __syncthreads();
    if (sh_count < p.nt && threadIdx.x == 0) atomicOr(err, 1);
    const uint32_t row = ((uint32_t)b * p.C + c) * p.ntp * 4;  // byte offset of the channel's row
    if (r < nsplit) {
      float acc = 0.f;
      for (int g0 = r; g0 < nq; g0 += kQuads * nsplit) {
        float bsum = 0.f;
        bool miss = true;
        for (int tries = 0; miss && tries < kSpinLimit; ++tries) {
          if (tries > 0) __builtin_amdgcn_s_sleep(8);
          // memory may have changed since the last try: the loads below are
          // not to be merged with those of the previous try
          asm volatile("" ::: "memory");
          uint4 v[kQuads];
#pragma unroll
          for (int q = 0; q < kQuads; ++q) {
            const uint32_t g = (uint32_t)min(g0 + q * nsplit, nq - 1);
            v[q] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, row + g * 16, 0, kSysCoherent));
          }
          miss = false;
          bsum = 0.f;
#pragma unroll
          for (int q = 0; q < kQuads; ++q) {
            const int j = 4 * (g0 + q * nsplit);
            const uint32_t e[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              if (j + u < p.nt) {
                miss |= e[u] == kSentinel;
                bsum += __uint_as_float(e[u]);
              }
            }
          }
        }
        if (miss) atomicOr(err, 1);
        acc += bsum;
      }
      red[threadIdx.x] = acc;
    }
    __syncthreads();
    if (threadIdx.x < p.C) {
      float sum = 0.f;
      for (int q = 0; q < nsplit; ++q) sum += red[q * p.C + threadIdx.x];
      dl[threadIdx.x] = sum / (float)p.HW;
    }
    __syncthreads();

    // per expert: g, tau, then the maximum and the log-partition of w / tau.
    // The image's rows of tau and lse are rebased here (the empty asm keeps
    // the compiler from precomputing per-lane addresses for every image,
    // which would not fit in registers).
    float* taub = tau + (int64_t)b * p.R;
    float* lseb = lse + (int64_t)b * p.R;
    asm volatile("" : "+s"(taub), "+s"(lseb));
    auto finish = [&](int o, float g, float t, float m, float z) {
      (void)g;
      if (o < p.R && gl == 0) {
        publish(taub + o, t);
        publish(lseb + o, m + logf(z));
      }
    };
    if (one) {
      // the kGatePass passes side by side, so that their lane reductions overlap
      float g[kGatePass], tq[kGatePass], m[kGatePass], z[kGatePass];
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) {
        const int o = threadIdx.x / p.gsz + q * gpp;
        g[q] = (o < p.R && gl < p.k) ? pa[q] * dl[ps[q]] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) g[q] = group_sum(g[q], p.gsz) + pc[q];
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) {
        const int o = threadIdx.x / p.gsz + q * gpp;
        tq[q] = softplusf(g[q]) + 1e-3f;
        m[q] = (o < p.R && gl < p.k) ? pw[q] / tq[q] : -INFINITY;
      }
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) m[q] = group_max(m[q], p.gsz);
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) {
        const int o = threadIdx.x / p.gsz + q * gpp;
        z[q] = (o < p.R && gl < p.k) ? expf(pw[q] / tq[q] - m[q]) : 0.f;
      }
#pragma unroll
      for (int q = 0; q < kGatePass; ++q) z[q] = group_sum(z[q], p.gsz);
#pragma unroll
      for (int q = 0; q < kGatePass; ++q)
        if (q < npass) finish(threadIdx.x / p.gsz + q * gpp, g[q], tq[q], m[q], z[q]);
    }
    for (int q = one ? kGatePass : 0; q < npass; ++q) {
      const int o = threadIdx.x / p.gsz + q * gpp;
      const bool active = o < p.R;
      const int oc = min(o, p.R - 1);
      float g = 0.f;
      for (int e = 0; e < p.epl; ++e) {
        const int i = gl + e * p.gsz;
        if (active && i < p.k) g += ga[(int64_t)oc * p.k + i] * dl[s[(int64_t)oc * p.k + i]];
      }
      g = group_sum(g, p.gsz) + gc[oc];
      const float t = softplusf(g) + 1e-3f;
      float m = -INFINITY;
      for (int e = 0; e < p.epl; ++e) {
        const int i = gl + e * p.gsz;
        if (active && i < p.k) m = fmaxf(m, w[(int64_t)oc * p.k + i] / t);
      }
      m = group_max(m, p.gsz);
      float z = 0.f;
      for (int e = 0; e < p.epl; ++e) {
        const int i = gl + e * p.gsz;
        if (active && i < p.k) z += expf(w[(int64_t)oc * p.k + i] / t - m);
      }
      z = group_sum(z, p.gsz);
      finish(o, g, t, m, z);
    }
    __syncthreads();  // red and dl are reused by the next image
  }
}

// y[o][p0 + 4 l .. +3] of one routed expert from lane l of a quarter wave: K
// (or kq, when K == 0) support entries, each a 16-byte read of the LDS tile at
// the entry's 16-bit byte offset plus the lane's own; offsets and
// coefficients read four at a time.  Padding entries have coefficient 0.
template <int K>
__device__ __forceinline__ float4 mix_expert(const uint16_t* ofs, const float* al, const char* base, int kq) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  const int n = K > 0 ? K : kq;
#pragma unroll 1
  for (int i = 0; i < n; i += 4) {
    const uint2 of = *reinterpret_cast<const uint2*>(ofs + i);
    const float4 a = *reinterpret_cast<const float4*>(al + i);
    const float4 v0 = *reinterpret_cast<const float4*>(base + (of.x & 0xffffu));
    const float4 v1 = *reinterpret_cast<const float4*>(base + (of.x >> 16));
    const float4 v2 = *reinterpret_cast<const float4*>(base + (of.y & 0xffffu));
    const float4 v3 = *reinterpret_cast<const float4*>(base + (of.y >> 16));
#define MOCE_FMA4(A, V) \
    acc.x = fmaf(A, V.x, acc.x); acc.y = fmaf(A, V.y, acc.y); acc.z = fmaf(A, V.z, acc.z); acc.w = fmaf(A, V.w, acc.w)
    MOCE_FMA4(a.x, v0); MOCE_FMA4(a.y, v1); MOCE_FMA4(a.z, v2); MOCE_FMA4(a.w, v3);
#undef MOCE_FMA4
  }
  return acc;
}

__device__ __forceinline__ uint2 pack_bf16x4(float4 v) {
  return make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
}

template <int K>
__global__ void __launch_bounds__(kThreads, 2 * kPerCU)
k_fused_nchw(FusedArgs p, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, float* __restrict__ part,
             float* __restrict__ tau, float* __restrict__ lse, int* __restrict__ arrive, int* __restrict__ err,
             const int32_t* __restrict__ s, const float* __restrict__ w, const float* __restrict__ ga,
             const float* __restrict__ gc, const int32_t* __restrict__ U) {
  extern __shared__ __align__(16) unsigned char smem[];
  const LdsLayout ll = lds_layout(p.C, p.R, p.kq);
  float* tile = reinterpret_cast<float*>(smem);                    // [C][kTT]
  float* alpha = reinterpret_cast<float*>(smem + ll.alpha);        // [R][kq], gate scratch
  uint16_t* sofs = reinterpret_cast<uint16_t*>(smem + ll.sofs);    // [R][kq]
  float2* tl = reinterpret_cast<float2*>(smem + ll.tl);            // [R]
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int G = gridDim.x - p.ng;  // mixing workgroups
  const float kLog2e = 1.4426950408889634f;
  const int rkq = p.R * p.kq;
  if ((int)blockIdx.x >= G) {
    gate_service(p, blockIdx.x - G, p.ng, part, tau, lse, arrive, err, s, w, ga, gc, reinterpret_cast<float*>(smem));
    return;
  }
  // byte offsets of the support rows in the LDS tile (padding: row 0)
  for (int e = threadIdx.x; e < rkq; e += kThreads) {
    const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
    const int32_t sv = s[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)];
    sofs[e] = (uint16_t)((i < p.k ? sv : 0) * kRowBytes);
  }
  // logits of the (expert, entry) pairs e = threadIdx.x + q * kThreads of the
  // [R][kq] layout (padding: -inf), kept in registers for the first kWSlots
  // passes of the coefficient loop
  float wr[kWSlots];
#pragma unroll
  for (int q = 0; q < kWSlots; ++q) {
    const int e = threadIdx.x + q * kThreads;
    const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
    const float v = w[min((int64_t)o * p.k + i, (int64_t)p.R * p.k - 1)];
    wr[q] = (e < rkq && i < p.k) ? v : -INFINITY;
  }

  // Publishes the channel sums of tile n (data in buf) at part[b][c][j].
  auto publish_tile = [&](int n, const uint4* buf) {
    const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
    float* pt = part + (int64_t)b * p.C * p.ntp + j;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (u * 64 < p.C) {
        const int c = (threadIdx.x >> 3) + u * 64;
        const float rs = group8_sum(tile_valid(p, n, u) ? sum8_bf16(buf[u]) : 0.f);
        if ((threadIdx.x & 7) == 0 && c < p.C) publish(pt + (int64_t)c * p.ntp, rs);
      }
    }
  };

  // Widens tile data into the LDS tile (positions past the end of the image
  // hold copies of earlier data; no output is stored for them).
  auto store_tile = [&](const uint4* buf) {
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
  };

  // One step with tile n in LDS and the data of tile n + G (if any) in nxt:
  // publish n + G, obtain the image's temperatures, start the loads of
  // n + 2G into spare, build the coefficients, mix.  Returns false after the
  // workgroup's last tile; otherwise tile n + G is in LDS on return.
  auto step = [&](int n, uint4* nxt, uint4* spare) -> bool {
    const int b = n / p.nt, j = n - (n / p.nt) * p.nt;
    const int n1 = n + G, n2 = n + 2 * G;
    if (!p.gated) {
      if (n1 < p.ntiles) publish_tile(n1, nxt);
      // every wave has issued its channel sums of n + G: count the tile (no
      // return value, so nothing waits for it)
      __syncthreads();
      if (n1 < p.ntiles && threadIdx.x == 0)
        __hip_atomic_fetch_add(arrive + n1 / p.nt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    // one lane waits for the image's gate (on the last value the service
    // publishes, with long pauses, to keep the polling traffic small); then
    // every lane reads its own two values, which are normally there already
    if (threadIdx.x == 0) {
      const uint32_t* last = reinterpret_cast<const uint32_t*>(lse + (int64_t)b * p.R + p.R - 1);
      for (int tries = 0; tries < kSpinLimit; ++tries) {
        if (__hip_atomic_load(last, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != kSentinel) break;
        __builtin_amdgcn_s_sleep(8);
      }
    }
    __syncthreads();
    if (threadIdx.x < p.R) {
      const int o = threadIdx.x;
      const float t = await_value(tau + (int64_t)b * p.R + o, err);
      const float l = await_value(lse + (int64_t)b * p.R + o, err);
      tl[o] = make_float2(kLog2e / t, -l * kLog2e);
    }
    __syncthreads();
    // the loads of n + 2G start once the temperatures are in hand, so that
    // polling for those never waits for these loads
    if (n2 < p.ntiles) issue_tile(p, x, n2, spare);
    // coefficients exp2(w * log2e / tau - lse * log2e) (padding: logit -inf, coefficient 0)
#pragma unroll
    for (int q = 0; q < kWSlots; ++q) {
      const int e = threadIdx.x + q * kThreads;
      if (e < rkq) {
        const float2 sc = tl[e / p.kq];
        alpha[e] = __builtin_amdgcn_exp2f(fmaf(wr[q], sc.x, sc.y));
      }
    }
    for (int e = threadIdx.x + kWSlots * kThreads; e < rkq; e += kThreads) {
      const int o = e / p.kq, i = e - (e / p.kq) * p.kq;
      const float lg = i < p.k ? w[(int64_t)o * p.k + i] : -INFINITY;
      const float2 sc = tl[o];
      alpha[e] = __builtin_amdgcn_exp2f(fmaf(lg, sc.x, sc.y));
    }
    __syncthreads();

    const int p0 = j * kTT;
    const int valid = min(kTT, p.HW - p0);
    const int gq = lane >> 4, l4 = lane & 15;
    const char* base = reinterpret_cast<const char*>(tile) + l4 * 16;
    uint16_t* yb = y + (int64_t)b * p.E * p.HW + p0 + l4 * 4;
    const bool store = l4 * 4 < valid;  // H*W is a multiple of 8: all four positions or none
    for (int o0 = 4 * wv; o0 <= p.R; o0 += 4 * kWaves) {
      const int o = o0 + gq;  // o == R is the residual output, channel E-1
      if (o < p.R) {
        const float4 acc = mix_expert<K>(sofs + o * p.kq, alpha + o * p.kq, base, p.kq);
        if (store) *reinterpret_cast<uint2*>(yb + (int64_t)o * p.HW) = pack_bf16x4(acc);
      } else if (o == p.R) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int u = 0; u < p.nU; ++u) {
          const float4 v = *reinterpret_cast<const float4*>(base + U[u] * kRowBytes);
          acc.x += v.x;
          acc.y += v.y;
          acc.z += v.z;
          acc.w += v.w;
        }
        if (p.nU > 0) {
          const float inv = (float)p.nU;
          acc = make_float4(acc.x / inv, acc.y / inv, acc.z / inv, acc.w / inv);
        }
        if (store) *reinterpret_cast<uint2*>(yb + (int64_t)p.R * p.HW) = pack_bf16x4(acc);
      }
    }
    if (n1 >= p.ntiles) return false;
    __syncthreads();  // the LDS tile and the coefficients are overwritten next
    store_tile(nxt);
    __syncthreads();
    return true;
  };

  int n = blockIdx.x;
  if (n >= p.ntiles) return;
  uint4 bufa[4], bufb[4];
  issue_tile(p, x, n, bufa);
  if (n + G < p.ntiles) issue_tile(p, x, n + G, bufb);
  if (!p.gated) publish_tile(n, bufa);
  store_tile(bufa);
  __syncthreads();
  if (!p.gated && threadIdx.x == 0)
    __hip_atomic_fetch_add(arrive + n / p.nt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  // two steps per trip, so that the two register buffers trade roles
  // without being copied
  for (;;) {
    if (!step(n, bufb, bufa)) break;
    n += G;
    if (!step(n, bufa, bufb)) break;
    n += G;
  }
}

// Per-call set-up: sentinels, tile counts and the error word.
__global__ void k_fused_fill(FusedArgs p, float* part, float* tau, float* lse, int* arrive, int* err) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float sent = __uint_as_float(kSentinel);
  const int64_t np = (int64_t)p.B * p.C * p.ntp, nr = (int64_t)p.B * p.R;
  for (int64_t i = i0; i < np; i += stride) part[i] = sent;
  for (int64_t i = i0; i < nr; i += stride) {
    tau[i] = sent;
    lse[i] = sent;
  }
  for (int64_t i = i0; i < p.B; i += stride) arrive[i] = 0;
  if (i0 == 0) err[0] = 0;
}

int rounded_k(const Shape& sh) { return (sh.k + 7) & ~7; }

int64_t tiles_per_image(const Shape& sh) { return (sh.HW + kTT - 1) / kTT; }

using FusedKernel = void (*)(FusedArgs, const uint16_t*, uint16_t*, float*, float*, float*, int*, int*,
                             const int32_t*, const float*, const float*, const float*, const int32_t*);

FusedKernel pick_kernel(const Shape& sh) {
  const int kq = rounded_k(sh);
  return kq == 32 ? k_fused_nchw<32> : kq == 64 ? k_fused_nchw<64> : k_fused_nchw<0>;
}

// Workgroups of the fused kernel that fit on the device at once, cached per
// device (the value depends only on the device and the kernel's resources).
std::atomic<int> g_resident[kMaxDevices][3];

int resident_workgroups(const Shape& sh, size_t lds) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  const int kq = rounded_k(sh);
  const int slot = kq == 32 ? 0 : kq == 64 ? 1 : 2;
  const int cached = g_resident[dev][slot].load(std::memory_order_relaxed);
  if (cached > 0) return cached;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 0;
  const FusedKernel kern = pick_kernel(sh);
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                          kMaxLds) != hipSuccess)
    return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern), kThreads,
                                                   kMaxLds) != hipSuccess ||
      per_cu <= 0)
    return 0;
  (void)lds;
  const int n = cus * std::min(per_cu, kPerCU);
  g_resident[dev][slot].store(n, std::memory_order_relaxed);
  return n;
}

int gate_group(int kq) {
  int g = 8;
  while (g < kq && g < 64) g <<= 1;
  return g;
}

}  // namespace

size_t fused_lds_bytes(const Shape& sh) { return lds_layout((int)sh.C, sh.R, rounded_k(sh)).total; }

size_t fused_partial_floats(const Shape& sh) { return (size_t)sh.B * sh.C * ((tiles_per_image(sh) + 3) & ~3); }

bool fused_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1 || sh.R > kThreads) return false;
  if (sh.HW % 8 != 0 || sh.HW < kTT || sh.C > 256 || tiles_per_image(sh) > 256) return false;
  if (sh.B * tiles_per_image(sh) > INT32_MAX / 4) return false;
  if (fused_partial_floats(sh) * 4 > (size_t)INT32_MAX) return false;  // offsets of the 32-bit buffer loads
  return fused_lds_bytes(sh) <= (size_t)kMaxLds;
}

bool fused_runnable(const Shape& sh) {
  if (!fused_eligible(sh)) return false;
  const int64_t nt = tiles_per_image(sh);
  const int ng = (int)std::min<int64_t>(sh.B, kGateWorkgroups);
  const int mixers = (int)std::min<int64_t>(resident_workgroups(sh, fused_lds_bytes(sh)) - ng, sh.B * nt);
  return mixers > 0 && (mixers >= nt || mixers >= sh.B * nt);
}

hipError_t launch_fused(const Shape& sh, const void* x, const int32_t* s, const float* w,
                        const moce_gate_params& g, const int32_t* U, int nU, void* y, const FusedWs& ws,
                        bool gated, hipStream_t st, bool* launched) {
  *launched = false;
  FusedArgs p;
  p.gated = gated ? 1 : 0;
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
  p.ntp = (p.nt + 3) & ~3;
  p.gsz = gate_group(p.kq);
  p.epl = (p.kq + p.gsz - 1) / p.gsz;

  const size_t lds = fused_lds_bytes(sh);
  const int resident = resident_workgroups(sh, lds);
  p.ng = gated ? 0 : (int)std::min<int64_t>(sh.B, kGateWorkgroups);
  const int mixers = std::min(resident - p.ng, p.ntiles);
  // every tile of an image must be held by a different resident workgroup
  if (mixers <= 0 || (mixers < p.nt && mixers < p.ntiles)) return hipSuccess;
  const int grid = mixers + p.ng;

  hipError_t e = hipSuccess;
  if (!gated) {
    const int64_t work = std::max<int64_t>((int64_t)p.B * p.C * p.ntp, sh.B * sh.R);
    const int64_t fill_blocks = std::min<int64_t>(std::max<int64_t>((work + 255) / 256, 1), 1024);
    hipLaunchKernelGGL(k_fused_fill, dim3((unsigned)fill_blocks), dim3(256), 0, st, p, ws.part, ws.tau, ws.lse,
                       ws.arrive, ws.err);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  FusedKernel kern = pick_kernel(sh);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  uint16_t* yp = static_cast<uint16_t*>(y);
  float* part = ws.part;
  float* tau = ws.tau;
  float* lse = ws.lse;
  int* arrive = ws.arrive;
  int* err = ws.err;
  const float* ga = g.a;
  const float* gc = g.c;
  void* args[] = {&p, &xp, &yp, &part, &tau, &lse, &arrive, &err, &s, &w, &ga, &gc, &U};
  if (gated) {
    // no workgroup waits for another: an ordinary launch (a cooperative one
    // costs several microseconds on each side)
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, st, p, xp, yp, part, tau, lse, arrive, err,
                       s, w, ga, gc, U);
    e = hipGetLastError();
  } else {
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3((unsigned)grid), dim3(kThreads), args,
                                   (unsigned)lds, st);
  }
  if (e == hipSuccess) *launched = true;
  return e;
}

}  // namespace moce

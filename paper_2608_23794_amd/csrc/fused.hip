// Fused forward for NCHW bfloat16 inputs: pooling, temperatures and mixing of
// every image in one persistent launch, so that the gather reads an image from
// the L2 of the XCD that has just pooled it rather than from HBM a second time.
//
// Work items.  Image b owns P pool items (8 channel planes each) and M mix
// items (one tile of 128 positions each).  Images are split over eight queues,
// b -> b % 8, and workgroup w serves queue w % 8, so the workgroups of a queue
// run on one XCD and share its L2.  A queue hands out tickets in the order
//   P(0) P(1) | P(2) M(0) | P(3) M(1) | ... | M(n-2) | M(n-1),
// so an image's mix items are claimed two images after its pool items.
//
// Mix tiles.  A tile holds all C (<= 256) channels x 128 positions as float32
// in LDS.  Lanes own 2 consecutive positions; each support entry costs one
// 8-byte LDS read and two FMAs, with the support row indices in scalar
// registers (scalar loads of the read-only support table, fully unrolled for
// the common support sizes) and the coefficients broadcast from LDS.
//
// Software pipeline.  The global loads of the next item (a pool item or a
// tile) are issued into registers before the current tile is mixed, and the
// next ticket is claimed one item ahead, so memory latency overlaps with the
// mixing arithmetic.
//
// Hand-off without fences.  Descriptors, temperatures and log-partitions
// start as a sentinel NaN (written by the fill kernel) and are published with
// system-scope stores; consumers poll them with system-scope loads.  Each
// value is its own ready flag, so no ordering between locations is needed and
// no acquire (which would invalidate the L2 holding the image) is issued.  The
// last pool item of an image (counted with an atomic add) waits for the
// image's descriptors, evaluates the gate of every expert and publishes tau
// and lse.
//
// Progress.  An item only waits for values published by items with smaller
// tickets of its own queue: a mix item for its image's gate, the gate for the
// image's pool items, which have all finished by the time the last of them
// counts itself.  The item a workgroup holds claimed but unstarted always has
// a larger ticket than the item it is working on, so the waiting item with the
// smallest ticket always depends only on running or finished work.  Every wait
// is in addition bounded (kSpinLimit polls); one that runs out sets err[0] and
// the kernel still terminates.
#include <algorithm>

#include "moce_internal.h"

namespace moce {
namespace {

constexpr uint32_t kSentinel = 0x7FC0DEADu;
constexpr int kQueues = 8;
constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTT = 128;           // positions per tile
constexpr int kPoolPlanes = 8;     // planes per pool item (two waves per plane)
constexpr int kSpinLimit = 1 << 22;
constexpr int kRowBytes = kTT * 4;

struct FusedArgs {
  const uint16_t* x;
  uint16_t* y;
  float* d;         // [B][C]    sentinel-filled
  float* tau;       // [B][R]    sentinel-filled
  float* lse;       // [B][R]    sentinel-filled
  int* pool_done;   // [B]       zeroed
  int* tickets;     // [kQueues] zeroed
  int* err;         // [1]       zeroed
  int B, C, HW, E, R, k, kp, nU;  // kp: k rounded up to a multiple of 4
  int P, M;
};

// Read-only tables.  They reach the kernel as separate __restrict__ arguments,
// which lets uniform accesses compile to scalar loads.
struct Tables {
  const int32_t* s;    // [R][k] canonical supports
  const float* w;      // [R][k] canonical logits
  const float* ga;     // [R][k] gate slopes
  const float* gc;     // [R]    gate offsets
  const int32_t* U;    // [nU] uncovered channels, ascending
};

__device__ __forceinline__ void publish(float* p, float v) {
  uint32_t u = __float_as_uint(v);
  if (u == kSentinel) u = 0x7FC00000u;  // never publish the sentinel itself
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ float await_value(const float* p, int* err) {
  const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
  uint32_t u = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  for (int n = 0; u == kSentinel && n < kSpinLimit; ++n) {
    __builtin_amdgcn_s_sleep(2);
    u = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (u == kSentinel) atomicOr(err, 1);
  return __uint_as_float(u);
}

// One relaxed system-scope load of a published value (may still be the sentinel).
__device__ __forceinline__ uint32_t peek_value(const float* p) {
  return __hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ float sum8_bf16(uint4 v) {
  return ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
         ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
}

struct Item {
  int img;   // index of the image within the queue
  int pool;  // pool item index, or -1
  int mix;   // mix item (tile) index, or -1
};

// Decodes ticket t of a queue of n images (order in the header comment).
__device__ __forceinline__ Item decode_ticket(int t, int n, int P, int M) {
  constexpr int kAhead = 2;
  Item it{0, -1, -1};
  const int head = min(n, kAhead);
  if (t < head * P) {
    it.img = t / P;
    it.pool = t - it.img * P;
    return it;
  }
  t -= head * P;
  const int full_steps = n - head;  // steps that still carry pool items
  if (t < full_steps * (P + M)) {
    const int step = t / (P + M);
    const int r = t - step * (P + M);
    if (r < P) {
      it.img = step + kAhead;
      it.pool = r;
    } else {
      it.img = step;
      it.mix = r - P;
    }
    return it;
  }
  t -= full_steps * (P + M);
  it.img = full_steps + t / M;
  it.mix = t - (t / M) * M;
  return it;
}

// Issues the global loads of one item into buf (4 x 16 bytes per thread).
// Pool item: waves 2j and 2j+1 read the two halves of plane j (first 256
// vectors of each half; longer planes are finished in pool_chunk).  Mix
// item: the C x 128 bf16 block of the tile (C <= 256).  Lanes past the data
// load a clamped, in-bounds address and keep zeros, so every load is a plain
// 16-byte global load (a conditional load would become a generic one).
__device__ __forceinline__ void issue_chunk(const FusedArgs& p, const Item& it, int b, int lane, int wv,
                                            uint4* buf, uint32_t* tl_pre) {
  const uint4 z = make_uint4(0, 0, 0, 0);
  if (it.pool >= 0) {
    const int plane = it.pool * kPoolPlanes + (wv >> 1);
    const int VP = p.HW / 8;
    const int half = (VP + 1) / 2;
    const int v0 = (wv & 1) * half;
    const int v1 = min(VP, v0 + half);
    const uint4* pl = reinterpret_cast<const uint4*>(p.x + ((int64_t)b * p.C + min(plane, p.C - 1)) * p.HW);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int v = v0 + lane + 64 * u;
      const uint4 t = pl[min(v, v1 - 1)];
      buf[u] = (plane < p.C && v < v1) ? t : z;
    }
  } else {
    const int p0 = it.mix * kTT;
    const int vvalid = min(kTT, p.HW - p0) / 8;
    const uint16_t* xb = p.x + (int64_t)b * p.C * p.HW + p0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = threadIdx.x + u * kThreads;
      const int c = idx >> 4, qv = idx & 15;
      const uint4 t =
          *reinterpret_cast<const uint4*>(xb + (int64_t)min(c, p.C - 1) * p.HW + min(qv, vvalid - 1) * 8);
      buf[u] = (c < p.C && qv < vvalid) ? t : z;
    }
    // the image's temperature and log-partition for expert threadIdx.x, if
    // already published (re-polled at staging otherwise)
    if (threadIdx.x < p.R) {
      tl_pre[0] = peek_value(p.tau + (int64_t)b * p.R + threadIdx.x);
      tl_pre[1] = peek_value(p.lse + (int64_t)b * p.R + threadIdx.x);
    }
  }
}

// Descriptor of the 8 planes of a pool item, from buf (plus the tail of planes
// longer than 4096 positions), published per plane.
__device__ __forceinline__ void pool_chunk(const FusedArgs& p, const Item& it, int b, int lane, int wv,
                                           const uint4* buf, float* part) {
  const int plane = it.pool * kPoolPlanes + (wv >> 1);
  float sum = 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) sum += sum8_bf16(buf[u]);
  const int VP = p.HW / 8;
  const int half = (VP + 1) / 2;
  const int v0 = (wv & 1) * half;
  const int v1 = min(VP, v0 + half);
  if (plane < p.C && v0 + 256 < v1) {
    const uint4* pl = reinterpret_cast<const uint4*>(p.x + ((int64_t)b * p.C + plane) * p.HW);
    for (int v = v0 + 256 + lane; v < v1; v += 64) sum += sum8_bf16(pl[v]);
  }
  sum = wave_sum(sum);
  if (lane == 0) part[wv] = sum;
  __syncthreads();
  if (threadIdx.x < kPoolPlanes) {
    const int pl = it.pool * kPoolPlanes + threadIdx.x;
    if (pl < p.C)
      publish(p.d + (int64_t)b * p.C + pl, (part[2 * threadIdx.x] + part[2 * threadIdx.x + 1]) / (float)p.HW);
  }
}

// The gate of every expert of image b (run by the image's last pool item).
__device__ __forceinline__ void gate_image(const FusedArgs& p, const Tables& tb, int b, int lane, int wv, float* dl) {
  for (int c = threadIdx.x; c < p.C; c += kThreads) dl[c] = await_value(p.d + (int64_t)b * p.C + c, p.err);
  __syncthreads();
  for (int o = wv; o < p.R; o += kWaves) {
    const int32_t* so = tb.s + (int64_t)o * p.k;
    const float* ao = tb.ga + (int64_t)o * p.k;
    const float* wo = tb.w + (int64_t)o * p.k;
    float g = 0.f;
    for (int i = lane; i < p.k; i += 64) g += ao[i] * dl[so[i]];
    g = wave_sum(g) + tb.gc[o];
    const float t = softplusf(g) + 1e-3f;
    float m = -INFINITY;
    for (int i = lane; i < p.k; i += 64) m = fmaxf(m, wo[i] / t);
    m = wave_max(m);
    float z = 0.f;
    for (int i = lane; i < p.k; i += 64) z += expf(wo[i] / t - m);
    z = wave_sum(z);
    if (lane == 0) {
      publish(p.tau + (int64_t)b * p.R + o, t);
      publish(p.lse + (int64_t)b * p.R + o, m + logf(z));
    }
  }
}

// y[o][p0 + 2 lane .. +1] of one routed expert: its K (or p.k, when K == 0)
// support rows, row indices from scalar loads, coefficients broadcast from LDS.
template <int K>
__device__ __forceinline__ float2 mix_expert(const int32_t* __restrict__ so, const float* ao, const float* trow,
                                             int k) {
  float a0 = 0.f, a1 = 0.f;
  if constexpr (K > 0) {
#pragma unroll 2
    for (int i = 0; i < K; i += 4) {
      const float4 al = *reinterpret_cast<const float4*>(ao + i);
      const float2 v0 = *reinterpret_cast<const float2*>(trow + so[i] * kTT);
      const float2 v1 = *reinterpret_cast<const float2*>(trow + so[i + 1] * kTT);
      const float2 v2 = *reinterpret_cast<const float2*>(trow + so[i + 2] * kTT);
      const float2 v3 = *reinterpret_cast<const float2*>(trow + so[i + 3] * kTT);
      a0 = fmaf(al.x, v0.x, a0); a1 = fmaf(al.x, v0.y, a1);
      a0 = fmaf(al.y, v1.x, a0); a1 = fmaf(al.y, v1.y, a1);
      a0 = fmaf(al.z, v2.x, a0); a1 = fmaf(al.z, v2.y, a1);
      a0 = fmaf(al.w, v3.x, a0); a1 = fmaf(al.w, v3.y, a1);
    }
  } else {
    int i = 0;
    for (; i + 4 <= k; i += 4) {
      const float4 al = *reinterpret_cast<const float4*>(ao + i);
      const float2 v0 = *reinterpret_cast<const float2*>(trow + so[i] * kTT);
      const float2 v1 = *reinterpret_cast<const float2*>(trow + so[i + 1] * kTT);
      const float2 v2 = *reinterpret_cast<const float2*>(trow + so[i + 2] * kTT);
      const float2 v3 = *reinterpret_cast<const float2*>(trow + so[i + 3] * kTT);
      a0 = fmaf(al.x, v0.x, a0); a1 = fmaf(al.x, v0.y, a1);
      a0 = fmaf(al.y, v1.x, a0); a1 = fmaf(al.y, v1.y, a1);
      a0 = fmaf(al.z, v2.x, a0); a1 = fmaf(al.z, v2.y, a1);
      a0 = fmaf(al.w, v3.x, a0); a1 = fmaf(al.w, v3.y, a1);
    }
    for (; i < k; ++i) {
      const float2 v = *reinterpret_cast<const float2*>(trow + so[i] * kTT);
      a0 = fmaf(ao[i], v.x, a0);
      a1 = fmaf(ao[i], v.y, a1);
    }
  }
  return make_float2(a0, a1);
}

template <int K>
__global__ void __launch_bounds__(kThreads)
k_fused_nchw(FusedArgs pa, const uint16_t* __restrict__ x, uint16_t* __restrict__ y, float* __restrict__ d,
             float* __restrict__ tau, float* __restrict__ lse, int* __restrict__ pool_done,
             int* __restrict__ tickets, int* __restrict__ err, const int32_t* __restrict__ s,
             const float* __restrict__ w, const float* __restrict__ ga, const float* __restrict__ gc,
             const int32_t* __restrict__ U) {
  // every pointer arrives as its own __restrict__ argument, so the compiler can
  // prove that no store of the kernel touches the read-only tables
  FusedArgs p = pa;
  p.x = x;
  p.y = y;
  p.d = d;
  p.tau = tau;
  p.lse = lse;
  p.pool_done = pool_done;
  p.tickets = tickets;
  p.err = err;
  const Tables tb{s, w, ga, gc, U};
  extern __shared__ __align__(16) unsigned char smem[];
  float* tile = reinterpret_cast<float*>(smem);                        // [C][kTT]
  float* alpha = tile + (size_t)p.C * kTT;                             // [R][kp]
  float2* tl = reinterpret_cast<float2*>(alpha + (size_t)p.R * p.kp);  // [R]
  float* dl = reinterpret_cast<float*>(tl + p.R);                      // [C]
  __shared__ float part[kWaves];
  __shared__ int sh_cur;
  __shared__ int sh_claim;
  __shared__ int sh_last;

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = blockIdx.x % kQueues;
  const int nimg = q < p.B ? (p.B - q + kQueues - 1) / kQueues : 0;
  const int items = nimg * (p.P + p.M);
  const float kLog2e = 1.4426950408889634f;

  if (threadIdx.x == 0) {
    sh_cur = atomicAdd(&p.tickets[q], 1);
    sh_claim = atomicAdd(&p.tickets[q], 1);
  }
  __syncthreads();
  // tickets are the same in every lane; readfirstlane lets the compiler know,
  // so everything derived from them lives in scalar registers
  int cur_t = __builtin_amdgcn_readfirstlane(sh_cur);
  int nxt_t = __builtin_amdgcn_readfirstlane(sh_claim);
  __syncthreads();

  uint4 buf[4];
  uint32_t tl_pre[2] = {kSentinel, kSentinel};
  if (cur_t < items) {
    const Item it = decode_ticket(cur_t, nimg, p.P, p.M);
    issue_chunk(p, it, q + kQueues * it.img, lane, wv, buf, tl_pre);
  }

  while (cur_t < items) {
    const Item it = decode_ticket(cur_t, nimg, p.P, p.M);
    const int b = q + kQueues * it.img;
    // the ticket after the next one is claimed now, while this item's loads land
    if (threadIdx.x == 0) sh_claim = atomicAdd(&p.tickets[q], 1);

    if (it.pool >= 0) {
      pool_chunk(p, it, b, lane, wv, buf, part);
      __syncthreads();
      // count this pool item, then issue the next item's loads before the
      // count comes back
      int done = 0;
      if (threadIdx.x == 0) done = atomicAdd(&p.pool_done[b], 1);
      if (nxt_t < items) {
        const Item nx = decode_ticket(nxt_t, nimg, p.P, p.M);
        issue_chunk(p, nx, q + kQueues * nx.img, lane, wv, buf, tl_pre);
      }
      if (threadIdx.x == 0) sh_last = (done == p.P - 1);
      __syncthreads();
      const bool last = __builtin_amdgcn_readfirstlane(sh_last) != 0;
      if (last) gate_image(p, tb, b, lane, wv, dl);
    } else {
      const int p0 = it.mix * kTT;
      const int valid = min(kTT, p.HW - p0);
      // the tile, widened to float32, and the image's temperatures (normally
      // already fetched with the tile)
      if (threadIdx.x < p.R) {
        const int o = threadIdx.x;
        const float t = tl_pre[0] != kSentinel ? __uint_as_float(tl_pre[0])
                                               : await_value(p.tau + (int64_t)b * p.R + o, p.err);
        const float l = tl_pre[1] != kSentinel ? __uint_as_float(tl_pre[1])
                                               : await_value(p.lse + (int64_t)b * p.R + o, p.err);
        tl[o] = make_float2(kLog2e / t, -l * kLog2e);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = threadIdx.x + u * kThreads;
        const int c = idx >> 4, qv = idx & 15;
        if (c < p.C) {
          float4* dst = reinterpret_cast<float4*>(tile + c * kTT + qv * 8);
          dst[0] = make_float4(bf16_lo(buf[u].x), bf16_hi(buf[u].x), bf16_lo(buf[u].y), bf16_hi(buf[u].y));
          dst[1] = make_float4(bf16_lo(buf[u].z), bf16_hi(buf[u].z), bf16_lo(buf[u].w), bf16_hi(buf[u].w));
        }
      }
      __syncthreads();
      // coefficients of every (expert, support entry), rows padded to kp with zeros
      const int rkp = p.R * p.kp;
      for (int e0 = threadIdx.x; e0 < rkp; e0 += 4 * kThreads) {
        float lg[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + u * kThreads;
          const int o = e / p.kp, i = e - o * p.kp;
          lg[u] = (e < rkp && i < p.k) ? w[(int64_t)o * p.k + i] : -INFINITY;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + u * kThreads;
          if (e < rkp) {
            const float2 sc = tl[e / p.kp];
            alpha[e] = __builtin_amdgcn_exp2f(fmaf(lg[u], sc.x, sc.y));  // exp2(-inf) = 0 for padding
          }
        }
      }
      __syncthreads();

      // the next item's loads fly while this tile is mixed
      if (nxt_t < items) {
        const Item nx = decode_ticket(nxt_t, nimg, p.P, p.M);
        issue_chunk(p, nx, q + kQueues * nx.img, lane, wv, buf, tl_pre);
      }

      const float* trow = tile + lane * 2;
      uint16_t* yb = p.y + (int64_t)b * p.E * p.HW + p0 + lane * 2;
      const bool store = lane * 2 < valid;  // H*W is a multiple of 8: both positions or neither
      for (int o = wv; o < p.R; o += kWaves) {
        const float2 acc = mix_expert<K>(s + (int64_t)o * p.k, alpha + o * p.kp, trow, p.k);
        if (store) *reinterpret_cast<uint32_t*>(yb + (int64_t)o * p.HW) = pack_bf16x2(acc.x, acc.y);
      }
      if (wv == p.R % kWaves) {  // the residual expert, channel E-1
        float a0 = 0.f, a1 = 0.f;
        for (int u = 0; u < p.nU; ++u) {
          const float2 v = *reinterpret_cast<const float2*>(trow + U[u] * kTT);
          a0 += v.x;
          a1 += v.y;
        }
        if (p.nU > 0) {
          a0 = a0 / (float)p.nU;
          a1 = a1 / (float)p.nU;
        }
        if (store) *reinterpret_cast<uint32_t*>(yb + (int64_t)p.R * p.HW) = pack_bf16x2(a0, a1);
      }
    }

    __syncthreads();
    cur_t = nxt_t;
    nxt_t = __builtin_amdgcn_readfirstlane(sh_claim);
    __syncthreads();  // sh_claim, part and the LDS tile are reused by the next item
  }
}

// Per-call set-up: sentinels and counters.
__global__ void k_fused_fill(FusedArgs p) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float sent = __uint_as_float(kSentinel);
  const int64_t nd = (int64_t)p.B * p.C, nt = (int64_t)p.B * p.R;
  for (int64_t i = i0; i < nd; i += stride) p.d[i] = sent;
  for (int64_t i = i0; i < nt; i += stride) {
    p.tau[i] = sent;
    p.lse[i] = sent;
  }
  for (int64_t i = i0; i < p.B; i += stride) p.pool_done[i] = 0;
  if (i0 < kQueues) p.tickets[i0] = 0;
  if (i0 == 0) p.err[0] = 0;
}

int rounded_k(const Shape& sh) { return (sh.k + 3) & ~3; }

}  // namespace

size_t fused_lds_bytes(const Shape& sh) {
  return (size_t)sh.C * kTT * 4 + (size_t)sh.R * rounded_k(sh) * 4 + (size_t)sh.R * 8 + (size_t)sh.C * 4;
}

size_t fused_plan_bytes(const Shape& sh) {
  (void)sh;
  return 0;
}

bool fused_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NCHW || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.HW % 8 != 0 || sh.HW < kTT || sh.C > 256 || sh.R > kThreads) return false;
  return fused_lds_bytes(sh) <= 160 * 1024 - 512;
}

hipError_t launch_fused(const Shape& sh, const void* x, const int32_t* s, const float* w,
                        const moce_gate_params& g, const int32_t* U, int nU, void* y, const FusedWs& ws,
                        hipStream_t st) {
  FusedArgs p;
  p.x = static_cast<const uint16_t*>(x);
  p.y = static_cast<uint16_t*>(y);
  p.d = ws.d;
  p.tau = ws.tau;
  p.lse = ws.lse;
  p.pool_done = ws.pool_done;
  p.tickets = ws.tickets;
  p.err = ws.err;
  p.B = (int)sh.B;
  p.C = (int)sh.C;
  p.HW = (int)sh.HW;
  p.E = sh.E;
  p.R = sh.R;
  p.k = sh.k;
  p.kp = rounded_k(sh);
  p.nU = nU;
  p.P = (p.C + kPoolPlanes - 1) / kPoolPlanes;
  p.M = (p.HW + kTT - 1) / kTT;

  const int64_t work = std::max<int64_t>(sh.B * sh.C, sh.B * sh.R);
  const int64_t fill_blocks = std::min<int64_t>(std::max<int64_t>((work + 255) / 256, 1), 1024);
  hipLaunchKernelGGL(k_fused_fill, dim3((unsigned)fill_blocks), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  int dev = 0;
  (void)hipGetDevice(&dev);
  int cus = 0;
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (cus <= 0) cus = 256;
  const int64_t grid = (cus + kQueues - 1) / kQueues * kQueues;  // one 1024-thread workgroup per CU
  const size_t lds = fused_lds_bytes(sh);
  auto kern = sh.k == 32 ? k_fused_nchw<32> : sh.k == 64 ? k_fused_nchw<64> : k_fused_nchw<0>;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, st, p, p.x, p.y, p.d, p.tau, p.lse,
                     p.pool_done, p.tickets, p.err, s, w, g.a, g.c, U);
  return hipGetLastError();
}

}  // namespace moce

// Channels-last mixing for small supports (k <= 16): the gather form of
// Sec. 3.3 Eq. 5 and Sec. 3.4 Eq. 6.
//
// With k small against C (k = 8 in the paper's ResNet-50 layers, against up to
// 2048 channels), the matrix-core form, whose products span every channel,
// does as much arithmetic as the dense projection itself; the gather does
// R k products per position and is bound by reading x.  x tiles are staged in
// LDS transposed, channel by channel, 8 positions per 16-byte row: a lane's
// one 16-byte read then serves one support entry at 8 positions at once, so
// the gather costs k reads per expert and octet of positions.  Row c sits at
// row c + c / 8: the eight rows one staging write spreads over then fall on
// distinct bank groups.
//
// A workgroup of 512 threads walks a contiguous range of position octets of
// the batch, about 32 KB of x per step.  The next step's 16-byte pieces are
// loaded into registers before the current step is mixed and written to the
// other LDS buffer after it, so the loads' latency overlaps the mixing.  A
// thread owns routed experts (one of up to 512 when E - 1 <= 512, the
// workgroup then holding several copies of the expert lanes that split the
// octets of a step; otherwise t and t + 512), holding their support channels
// in registers and their coefficients (reloaded when the image changes); it
// accumulates 8 positions per expert and writes y[b][p][e] with consecutive
// experts on consecutive lanes.  The residual output (the mean over U) of an
// octet is summed by one wave, lanes splitting U, and reduced by a
// reduce-scatter over the eight positions.
#include <algorithm>

#include "moce_internal.h"

namespace moce {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGThreads = 512;
constexpr int kGMaxK = 16;
constexpr int kGStepBytes = 32 * 1024;      // x bytes per step
constexpr int kGMaxC = 4096;                // two step buffers of 4608 16-byte rows and U: 152 KB of LDS

struct GatherArgs {
  const uint16_t* x;
  const float* alpha;    // [B][R][k]
  const int32_t* s;      // [R][k]
  const int32_t* U;
  uint16_t* y;
  int noct;              // position octets in the batch: B * ceil(HW / 8)
  int C, HW, E, R, k, nU, opi;   // opi: octets per image
  int ts;                // octets per step
  Epi ep;
};

__device__ __forceinline__ void acc8(float (&acc)[8], const u32x4 v, float c) {
  acc[0] += c * bf16_lo(v.x);
  acc[1] += c * bf16_hi(v.x);
  acc[2] += c * bf16_lo(v.y);
  acc[3] += c * bf16_hi(v.y);
  acc[4] += c * bf16_lo(v.z);
  acc[5] += c * bf16_hi(v.z);
  acc[6] += c * bf16_lo(v.w);
  acc[7] += c * bf16_hi(v.w);
}

__device__ __forceinline__ float epi(const Epi& ep, float v, float sc, float sf) {
  if (ep.scale) v = __builtin_fmaf(v, sc, sf);
  if (ep.relu) v = fmaxf(v, 0.f);
  return v;
}

// EPT: routed experts per thread; KK: support registers (k <= KK); NP: pieces
// per thread and step (ts C <= 512 NP)
template <int EPT, int KK, int NP>
__global__ void __launch_bounds__(kGThreads)
k_gather_nhwc(GatherArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = a.C, k = a.k, c8n = C >> 3;
  const int crow = C + c8n;                               // rows of one octet, with the spreading gaps
  const int sbytes = a.ts * crow * 16;                    // one step buffer: [ts][crow][8] bf16
  uint16_t* Ul = reinterpret_cast<uint16_t*>(lds + 2 * sbytes);

  const int o0 = (int)((int64_t)a.noct * blockIdx.x / gridDim.x);
  const int o1 = (int)((int64_t)a.noct * (blockIdx.x + 1) / gridDim.x);
  if (o0 >= o1) return;
  for (int i = tid; i < a.nU; i += kGThreads) Ul[i] = (uint16_t)a.U[i];

  // the experts of this thread and the octets of a step it mixes: with E - 1
  // <= 512 the workgroup holds G copies of the R64 expert lanes, copy g
  // taking octets g, g + G, ...
  const int R64 = EPT == 1 ? ((a.R + 63) & ~63) : kGThreads;
  const int G = kGThreads / R64;
  const int grp = tid / R64;
  const int e0 = tid - grp * R64;
  const bool mixer = grp < G && e0 < a.R;

  // support channels of this thread's experts, two 16-bit channels a register
  uint32_t ch[EPT][KK / 2];
  float sc[EPT], sf[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int e = min(e0 + j * kGThreads, a.R - 1);
#pragma unroll
    for (int i = 0; i < KK; i += 2) {
      const uint32_t lo = (uint32_t)a.s[(int64_t)e * k + min(i, k - 1)];
      const uint32_t hi = (uint32_t)a.s[(int64_t)e * k + min(i + 1, k - 1)];
      ch[j][i / 2] = lo | (hi << 16);
    }
    sc[j] = a.ep.scale ? a.ep.scale[e] : 1.f;
    sf[j] = a.ep.scale ? a.ep.shift[e] : 0.f;
  }
  float al[EPT][KK];
  int img = -1;

  // the pieces of this thread in every step: piece q = tid + 512 i is
  // position q % 8 of channel group (q / 8) % (C / 8) of the step's octet
  // (q / 8) / (C / 8); packed as octet << 16 | group << 3 | position
  const int pieces = a.ts * C;
  uint32_t pk[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = tid + i * kGThreads;
    const int r = q >> 3;
    const int t = r / c8n;
    pk[i] = q < pieces ? ((uint32_t)t << 16) | ((uint32_t)(r - t * c8n) << 3) | (uint32_t)(q & 7) : 0xffffffffu;
  }
  u32x4 pv[NP];
  // load the pieces of the step at octet oct0 (nst octets) into registers
  auto issue = [&](int oct0, int nst) {
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      pv[i] = u32x4{0u, 0u, 0u, 0u};
      const int t = (int)(pk[i] >> 16);
      if (pk[i] != 0xffffffffu && t < nst) {
        const int oc = oct0 + t;
        const int b = oc / a.opi;
        const int p = (oc - b * a.opi) * 8 + (int)(pk[i] & 7u);
        if (p < a.HW)
          pv[i] = __builtin_nontemporal_load(
              reinterpret_cast<const u32x4*>(a.x + ((int64_t)b * a.HW + p) * C + (pk[i] & 0xfff8u)));
      }
    }
  };
  // write them transposed: channel c of position q of octet t to byte
  // (t crow + c + c / 8) 16 + 2 q
  auto commit = [&](unsigned char* buf) {
    uint16_t* base = reinterpret_cast<uint16_t*>(buf);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if (pk[i] == 0xffffffffu) continue;
      const int t = (int)(pk[i] >> 16), g = (int)((pk[i] >> 3) & 0x1fffu), pos = (int)(pk[i] & 7u);
      uint16_t* dst = base + (t * crow + g * 9) * 8 + pos;
      const uint32_t w[4] = {pv[i].x, pv[i].y, pv[i].z, pv[i].w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        dst[(2 * h) * 8] = (uint16_t)(w[h] & 0xffffu);
        dst[(2 * h + 1) * 8] = (uint16_t)(w[h] >> 16);
      }
    }
  };

  const float inv = a.nU > 0 ? 1.f / (float)a.nU : 0.f;
  const int er = a.E - 1;
  const float rsc = a.ep.scale ? a.ep.scale[er] : 1.f, rsf = a.ep.scale ? a.ep.shift[er] : 0.f;

  int cur = 0;
  issue(o0, min(a.ts, o1 - o0));
  commit(lds);
  __syncthreads();
  for (int os = o0; os < o1; os += a.ts) {
    const int nst = min(a.ts, o1 - os);
    const bool more = os + a.ts < o1;
    if (more) issue(os + a.ts, min(a.ts, o1 - os - a.ts));
    const unsigned char* buf = lds + cur * sbytes;
    if (mixer && grp < nst) {
      // image and first position of octet os + grp, advanced by G octets
      int b = (os + grp) / a.opi;
      int pb = (os + grp - b * a.opi) * 8;
      for (int t = grp; t < nst; t += G) {
        if (b != img) {  // the image's coefficients of this thread's experts
          img = b;
#pragma unroll
          for (int j = 0; j < EPT; ++j) {
            const int e = min(e0 + j * kGThreads, a.R - 1);
#pragma unroll
            for (int i = 0; i < KK; ++i) al[j][i] = i < k ? a.alpha[((int64_t)b * a.R + e) * k + i] : 0.f;
          }
        }
        const unsigned char* tb = buf + t * crow * 16;
#pragma unroll
        for (int j = 0; j < EPT; ++j) {
          const int e = e0 + j * kGThreads;
          if (e >= a.R) break;
          float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int i = 0; i < KK; ++i) {
            if (i >= k) break;
            const int c = (int)((ch[j][i / 2] >> (16 * (i & 1))) & 0xffffu);
            acc8(acc, *reinterpret_cast<const u32x4*>(tb + (c + (c >> 3)) * 16), al[j][i]);
          }
          uint16_t* yp = a.y + ((int64_t)b * a.HW + pb) * a.E + e;
          if (pb + 8 <= a.HW) {
#pragma unroll
            for (int q = 0; q < 8; ++q) yp[(int64_t)q * a.E] = f32_to_bf16(epi(a.ep, acc[q], sc[j], sf[j]));
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q)
              if (pb + q < a.HW) yp[(int64_t)q * a.E] = f32_to_bf16(epi(a.ep, acc[q], sc[j], sf[j]));
          }
        }
        pb += 8 * G;
        while (pb >= a.opi * 8) {
          pb -= a.opi * 8;
          ++b;
        }
      }
    }
    // the residual outputs: wave w takes octets w, w + 8, ...; lanes split U,
    // then a reduce-scatter leaves position j's total in lane 8 j
    for (int t = wave; t < nst; t += kGThreads / kWave) {
      const int oc = os + t;
      const int b = oc / a.opi;
      const int pb = (oc - b * a.opi) * 8;
      float r1 = 0.f;
      if (a.nU > 0) {
        const unsigned char* tb = buf + t * crow * 16;
        float r[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int u = lane; u < a.nU; u += kWave) {
          const int c = Ul[u];
          acc8(r, *reinterpret_cast<const u32x4*>(tb + (c + (c >> 3)) * 16), 1.f);
        }
        const bool h5 = lane & 32, h4 = lane & 16, h3 = lane & 8;
        float r4[4], r2[2];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float send = h5 ? r[j] : r[j + 4];
          r4[j] = (h5 ? r[j + 4] : r[j]) + __shfl_xor(send, 32, kWave);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const float send = h4 ? r4[j] : r4[j + 2];
          r2[j] = (h4 ? r4[j + 2] : r4[j]) + __shfl_xor(send, 16, kWave);
        }
        r1 = (h3 ? r2[1] : r2[0]) + __shfl_xor(h3 ? r2[0] : r2[1], 8, kWave);
        r1 += __shfl_xor(r1, 4, kWave);
        r1 += __shfl_xor(r1, 2, kWave);
        r1 += __shfl_xor(r1, 1, kWave);
      }
      const int q = lane >> 3;
      if ((lane & 7) == 0 && pb + q < a.HW)
        a.y[((int64_t)b * a.HW + pb + q) * a.E + er] = f32_to_bf16(epi(a.ep, r1 * inv, rsc, rsf));
    }
    if (more) commit(lds + (cur ^ 1) * sbytes);
    __syncthreads();  // step buffer cur consumed; the next one written
    cur ^= 1;
  }
}

}  // namespace

bool gather_eligible(const Shape& sh) {
  if (sh.layout != MOCE_NHWC || sh.elem != MOCE_BF16 || sh.R < 1) return false;
  if (sh.k > kGMaxK || sh.C % 8 != 0 || sh.C > kGMaxC) return false;
  if (sh.R > (sh.k <= 8 ? 2 : 1) * kGThreads) return false;   // support and coefficient registers
  return sh.B * ((sh.HW + 7) / 8) < INT32_MAX / 2 && sh.B * sh.HW < INT32_MAX;
}

hipError_t launch_gather(const Shape& sh, const void* x, const int32_t* s, const float* alpha, const int32_t* U,
                         int nU, void* y, hipStream_t st, const Epi& ep) {
  GatherArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.alpha = alpha;
  a.s = s;
  a.U = U;
  a.y = static_cast<uint16_t*>(y);
  a.C = (int)sh.C;
  a.HW = (int)sh.HW;
  a.E = sh.E;
  a.R = sh.R;
  a.k = sh.k;
  a.nU = nU;
  a.opi = (int)((sh.HW + 7) / 8);
  a.noct = (int)(sh.B * a.opi);
  a.ts = std::max(1, std::min(a.opi, kGStepBytes / (16 * (a.C + a.C / 8))));
  a.ep = ep;
  const size_t lds = (size_t)2 * a.ts * (a.C + a.C / 8) * 16 + (size_t)sh.C * sizeof(uint16_t);
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess || cus <= 0)
    cus = 256;
  const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(a.noct, (int64_t)cus * 2));
  const bool two = sh.R > kGThreads;
  const bool wide = a.ts * a.C > 4 * kGThreads;   // more than 4 pieces per thread (C > 2048)
  using K = void (*)(GatherArgs);
  K k;
  if (sh.k <= 8)
    k = wide ? (two ? k_gather_nhwc<2, 8, 8> : k_gather_nhwc<1, 8, 8>)
             : (two ? k_gather_nhwc<2, 8, 4> : k_gather_nhwc<1, 8, 4>);
  else
    k = wide ? k_gather_nhwc<1, 16, 8> : k_gather_nhwc<1, 16, 4>;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kGThreads), lds, st, a);
  return hipGetLastError();
}

}  // namespace moce

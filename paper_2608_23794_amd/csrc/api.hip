// C ABI of libmoce: host-side validation, workspace layout and dispatch to
// the kernels of prepare.hip, pool.hip, gate.hip and mix.hip.  Every check that
// can fail on the host runs before anything is enqueued.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>

#include "moce_internal.h"

using moce::Shape;

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

moce_status check_desc(const moce_desc* d, Shape* sh) {
  if (!d) return MOCE_ERR_NULL;
  if (d->B < 1 || d->C < 1 || d->H < 1 || d->W < 1) return MOCE_ERR_SHAPE;
  if (d->E < 1 || (int64_t)d->E > d->C || d->k < 1 || (int64_t)d->k > d->C) return MOCE_ERR_SHAPE;
  if (d->x_dtype != MOCE_F32 && d->x_dtype != MOCE_BF16) return MOCE_ERR_DTYPE;
  if (d->y_dtype != d->x_dtype) return MOCE_ERR_DTYPE;
  if (d->layout != MOCE_NCHW && d->layout != MOCE_NHWC) return MOCE_ERR_LAYOUT;
  // index arithmetic: positions, channels and per-image element counts fit int32
  if (d->H > INT_MAX || d->W > INT_MAX || d->C > INT_MAX) return MOCE_ERR_UNSUPPORTED;
  const int64_t HW = d->H * d->W;
  if (d->H > INT_MAX / d->W) return MOCE_ERR_UNSUPPORTED;
  if (d->C > (int64_t)INT_MAX / HW) return MOCE_ERR_UNSUPPORTED;
  if (d->B > ((int64_t)1 << 40) / (d->C * HW)) return MOCE_ERR_UNSUPPORTED;
  if ((int64_t)d->E * d->k > INT_MAX) return MOCE_ERR_UNSUPPORTED;
  sh->B = d->B;
  sh->C = d->C;
  sh->HW = HW;
  sh->E = d->E;
  sh->R = d->E - 1;
  sh->k = d->k;
  sh->elem = d->x_dtype;
  sh->layout = d->layout;
  return MOCE_OK;
}

moce_status check_gate(const Shape& sh, const moce_gate_params* g) {
  if (!g) return MOCE_ERR_NULL;
  if (g->kind == MOCE_GATE_SOFTPLUS_LINEAR) {
    if (sh.R > 0 && (!g->a || !g->c)) return MOCE_ERR_NULL;
    return MOCE_OK;
  }
  if (g->kind == MOCE_GATE_MLP_SIGMOID) {
    if (sh.R > 0 && (!g->W1 || !g->b1 || !g->w2)) return MOCE_ERR_NULL;
    if (!std::isfinite(g->tau_min) || !std::isfinite(g->tau_max) || !std::isfinite(g->b2) ||
        g->tau_min <= 0.f || g->tau_max < g->tau_min)
      return MOCE_ERR_GATE;
    if (sh.k > 256) return MOCE_ERR_UNSUPPORTED;
    return MOCE_OK;
  }
  return MOCE_ERR_GATE;
}

moce_status device_status(hipError_t e) { return e == hipSuccess ? MOCE_OK : MOCE_ERR_DEVICE; }

size_t elem_bytes(const Shape& sh) { return sh.elem == MOCE_F32 ? 4 : 2; }

// Forward workspace: d [B][C], tau [B][R], the softmax statistics
// [3][B][R] (rt, m, rzs), and for NCHW the coefficients alpha [B][R][k];
// every region starts on a 256-byte boundary.
struct WsLayout {
  size_t d, tau, stats, alpha, sched, total;
};
// the forward's scheduled matrix-core mix: where gmix applies and no earlier
// path of forward_launch does
bool uses_gmix(const Shape& sh) {
  return !moce::mfmamix_eligible(sh) && !(sh.R > 0 && moce::tilemix_eligible(sh)) && !moce::gather_eligible(sh) &&
         moce::gmix_eligible(sh);
}

WsLayout ws_layout(const Shape& sh) {
  WsLayout l{};
  size_t off = 0;
  l.d = off;
  off += round_up((size_t)sh.B * sh.C * sizeof(float));
  l.tau = off;
  off += round_up((size_t)sh.B * sh.R * sizeof(float));
  l.stats = off;
  off += round_up((size_t)3 * sh.B * sh.R * sizeof(float));
  l.alpha = off;
  const bool gm = uses_gmix(sh);
  if ((sh.layout == MOCE_NCHW && !gm) || moce::gather_eligible(sh))
    off += round_up((size_t)sh.B * sh.R * sh.k * sizeof(float));
  l.sched = off;
  if (gm) off += round_up(moce::gmix_sched_bytes(sh));
  l.total = off;
  return l;
}

}  // namespace

extern "C" {

int moce_abi_version(void) { return 1; }

const char* moce_status_str(int status) {
  switch (status) {
    case MOCE_OK: return "MOCE_OK";
    case MOCE_ERR_NULL: return "MOCE_ERR_NULL: a required pointer is NULL";
    case MOCE_ERR_SHAPE: return "MOCE_ERR_SHAPE: invalid B, C, H, W, E or k";
    case MOCE_ERR_DTYPE: return "MOCE_ERR_DTYPE: unknown or mismatched element type";
    case MOCE_ERR_LAYOUT: return "MOCE_ERR_LAYOUT: unknown layout";
    case MOCE_ERR_SUPPORT: return "MOCE_ERR_SUPPORT: invalid support row";
    case MOCE_ERR_GATE: return "MOCE_ERR_GATE: invalid gate kind or parameters";
    case MOCE_ERR_WORKSPACE: return "MOCE_ERR_WORKSPACE: workspace missing or too small";
    case MOCE_ERR_ALIGN: return "MOCE_ERR_ALIGN: pointer not aligned";
    case MOCE_ERR_DEVICE: return "MOCE_ERR_DEVICE: HIP call or kernel launch failed";
    case MOCE_ERR_UNSUPPORTED: return "MOCE_ERR_UNSUPPORTED: shape exceeds a size limit";
    default: return "unknown moce_status";
  }
}

namespace {

moce_status support_prepare(const moce_desc* desc, const void* s, bool s16, const float* w, int32_t* s_out,
                            float* w_out, uint8_t* covered, int32_t* U, int32_t* info, int32_t* nU_host,
                            int32_t* bad_expert_host, hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  if (!covered || !U || !info || !nU_host || !bad_expert_host) return MOCE_ERR_NULL;
  if (sh.R > 0 && (!s || !w || !s_out || !w_out)) return MOCE_ERR_NULL;
  if (sh.C > (s16 ? (1 << 16) : (1 << 24)) || sh.k > 4096) return MOCE_ERR_UNSUPPORTED;
  if (sh.R > 0 && (s == static_cast<const void*>(s_out) || static_cast<const void*>(w) == w_out))
    return MOCE_ERR_NULL;
  hipError_t e = moce::launch_prepare(sh, s, s16, w, s_out, w_out, covered, U, info, stream);
  if (e != hipSuccess) return MOCE_ERR_DEVICE;
  int32_t host[2] = {0, 0};
  e = hipMemcpyAsync(host, info, sizeof host, hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return MOCE_ERR_DEVICE;
  e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return MOCE_ERR_DEVICE;
  *nU_host = host[0];
  *bad_expert_host = host[1];
  return host[1] >= 0 ? MOCE_ERR_SUPPORT : MOCE_OK;
}

}  // namespace

moce_status moce_support_prepare(const moce_desc* desc, const int32_t* s, const float* w,
                                 int32_t* s_out, float* w_out, uint8_t* covered, int32_t* U,
                                 int32_t* info, int32_t* nU_host, int32_t* bad_expert_host,
                                 hipStream_t stream) {
  return support_prepare(desc, s, false, w, s_out, w_out, covered, U, info, nU_host, bad_expert_host, stream);
}

moce_status moce_support_prepare16(const moce_desc* desc, const uint16_t* s, const float* w,
                                   int32_t* s_out, float* w_out, uint8_t* covered, int32_t* U,
                                   int32_t* info, int32_t* nU_host, int32_t* bad_expert_host,
                                   hipStream_t stream) {
  return support_prepare(desc, s, true, w, s_out, w_out, covered, U, info, nU_host, bad_expert_host, stream);
}

moce_status moce_pool(const moce_desc* desc, const void* x, float* d, hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  if (!x || !d) return MOCE_ERR_NULL;
  if (!aligned(x, 16) || !aligned(d, 4)) return MOCE_ERR_ALIGN;
  return device_status(moce::launch_pool(sh, x, d, stream));
}

moce_status moce_gate(const moce_desc* desc, const float* d, const int32_t* s, const float* w,
                      const moce_gate_params* gate, float* tau, float* alpha, hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  st = check_gate(sh, gate);
  if (st != MOCE_OK) return st;
  if (sh.R == 0) return MOCE_OK;
  if (!d || !s || !w || !tau) return MOCE_ERR_NULL;
  return device_status(moce::launch_gate(sh, d, s, w, *gate, tau, alpha, nullptr, stream));
}

moce_status moce_mix(const moce_desc* desc, const void* x, const int32_t* s, const float* alpha,
                     const int32_t* U, int32_t nU, void* y, hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  if (!x || !y) return MOCE_ERR_NULL;
  if (sh.R > 0 && (!s || !alpha)) return MOCE_ERR_NULL;
  if (nU < 0 || (int64_t)nU > sh.C) return MOCE_ERR_SHAPE;
  if (nU > 0 && !U) return MOCE_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return MOCE_ERR_ALIGN;
  if (moce::gather_eligible(sh))
    return device_status(moce::launch_gather(sh, x, s, alpha, U, nU, y, stream, moce::Epi{}));
  if (moce::mfmamix_eligible(sh))
    return device_status(moce::launch_mfmamix(sh, x, s, alpha, U, nU, y, stream));
  if (sh.R > 0 && moce::tilemix_eligible(sh))
    return device_status(moce::launch_tilemix(sh, x, s, alpha, U, nU, y, stream));
  return device_status(moce::launch_mix(sh, x, s, alpha, nullptr, nullptr, U, nU, y, stream));
}

moce_status moce_gate_mix(const moce_desc* desc, const void* x, const float* d, const int32_t* s, const float* w,
                          const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y,
                          hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  st = check_gate(sh, gate);
  if (st != MOCE_OK) return st;
  if (!moce::mfmamix_gate_fusable(sh, gate->kind)) return MOCE_ERR_UNSUPPORTED;
  if (!x || !y || !d || !s || !w) return MOCE_ERR_NULL;
  if (nU < 0 || (int64_t)nU > sh.C) return MOCE_ERR_SHAPE;
  if (nU > 0 && !U) return MOCE_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return MOCE_ERR_ALIGN;
  return device_status(moce::launch_mfmamix_gated(sh, x, s, w, d, gate->a, gate->c, U, nU, y, stream));
}

size_t moce_forward_workspace_bytes(const moce_desc* desc) {
  Shape sh;
  if (check_desc(desc, &sh) != MOCE_OK) return 0;
  return ws_layout(sh).total;
}

int moce_forward_path(const moce_desc* desc, int gate_kind) {
  Shape sh;
  const moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  if (gate_kind != MOCE_GATE_SOFTPLUS_LINEAR && gate_kind != MOCE_GATE_MLP_SIGMOID) return MOCE_ERR_GATE;
  // the order of forward_launch's tests
  if (moce::mfmamix_eligible(sh))
    return moce::mfmamix_gate_fusable(sh, gate_kind) ? MOCE_PATH_MFMA_GATE : MOCE_PATH_MFMA;
  if (sh.R > 0 && moce::tilemix_eligible(sh)) return MOCE_PATH_TILE;
  if (moce::gather_eligible(sh)) return MOCE_PATH_GATHER;
  if (moce::gmix_eligible(sh)) return MOCE_PATH_SCHEDULED;
  return MOCE_PATH_GENERIC;
}

}  // extern "C"

namespace {

// The host-side checks of the forward's arguments other than the workspace.
moce_status check_forward(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                          const moce_gate_params* gate, const int32_t* U, int32_t nU, const void* y, Shape* sh) {
  moce_status st = check_desc(desc, sh);
  if (st != MOCE_OK) return st;
  st = check_gate(*sh, gate);
  if (st != MOCE_OK) return st;
  if (!x || !y) return MOCE_ERR_NULL;
  if (sh->R > 0 && (!s || !w)) return MOCE_ERR_NULL;
  if (nU < 0 || (int64_t)nU > sh->C) return MOCE_ERR_SHAPE;
  if (nU > 0 && !U) return MOCE_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return MOCE_ERR_ALIGN;
  return MOCE_OK;
}

// The forward's launches on a validated call, with the workspace at `ws`
// (device memory of at least ws_layout(sh).total bytes, 256-byte aligned).
moce_status forward_launch(const Shape& sh, const void* x, const int32_t* s, const float* w,
                           const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y, void* ws,
                           hipStream_t stream, const moce::Epi& ep = moce::Epi{}) {
  const WsLayout l = ws_layout(sh);
  char* base = static_cast<char*>(ws);
  float* d = reinterpret_cast<float*>(base + l.d);
  float* tau = reinterpret_cast<float*>(base + l.tau);
  float* stats = reinterpret_cast<float*>(base + l.stats);
  float* alpha = (sh.layout == MOCE_NCHW && !uses_gmix(sh)) || moce::gather_eligible(sh)
                     ? reinterpret_cast<float*>(base + l.alpha)
                     : nullptr;

  // pooling reads x plane by plane (the order HBM serves best) and leaves it
  // in the infinity cache; the gate kernel writes tau and the coefficients;
  // the mix then reads x back from the cache
  if (moce::mfmamix_eligible(sh)) {
    hipError_t e = moce::launch_pool(sh, x, d, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    // k = 32 with the softplus-linear gate: the mix kernel evaluates the
    // gate itself, in the gate kernel's layout and operations
    if (moce::mfmamix_gate_fusable(sh, gate->kind))
      return device_status(moce::launch_mfmamix_gated(sh, x, s, w, d, gate->a, gate->c, U, nU, y, stream, ep));
    e = moce::launch_gate(sh, d, s, w, *gate, tau, alpha, nullptr, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    return device_status(moce::launch_mfmamix(sh, x, s, alpha, U, nU, y, stream, ep));
  }
  if (sh.R > 0 && moce::tilemix_eligible(sh)) {
    hipError_t e = moce::launch_pool(sh, x, d, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    e = moce::launch_gate(sh, d, s, w, *gate, tau, alpha, nullptr, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    e = moce::launch_tilemix(sh, x, s, alpha, U, nU, y, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    return device_status(moce::launch_epilogue(sh, y, ep, stream));
  }
  if (moce::gather_eligible(sh)) {
    // channels-last with small supports: pooling, the gate's coefficients,
    // then the gather, whose work scales with k
    hipError_t e = moce::launch_pool(sh, x, d, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    e = moce::launch_gate(sh, d, s, w, *gate, tau, alpha, nullptr, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    return device_status(moce::launch_gather(sh, x, s, alpha, U, nU, y, stream, ep));
  }
  if (moce::gmix_eligible(sh)) {
    // on the matrix cores: pooling with the support schedule (beside it for
    // channels-last x), the gate's softmax statistics, then the mix
    hipError_t e = moce::launch_pool_sched(sh, x, d, s, w, U, nU, base + l.sched, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    e = moce::launch_gate(sh, d, s, w, *gate, tau, nullptr, stats, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
    return device_status(moce::launch_gmix(sh, x, stats, nU, base + l.sched, y, stream, ep));
  }
  hipError_t e = moce::launch_pool(sh, x, d, stream);
  if (e != hipSuccess) return MOCE_ERR_DEVICE;
  if (sh.R > 0) {
    e = moce::launch_gate(sh, d, s, w, *gate, tau, alpha, alpha ? nullptr : stats, stream);
    if (e != hipSuccess) return MOCE_ERR_DEVICE;
  }
  e = moce::launch_mix(sh, x, s, alpha, w, stats, U, nU, y, stream);
  if (e != hipSuccess) return MOCE_ERR_DEVICE;
  return device_status(moce::launch_epilogue(sh, y, ep, stream));
}

// ---- the forward without a workspace argument ------------------------------
//
// Its workspace is this file-scope device array.  In host code the array's
// name is only a stand-in for the symbol, not a device address: the address
// comes from hipGetSymbolAddress, taken once per device with that device
// current, and only that address is ever handed to a kernel.
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
static_assert(kStaticScratchBytes == MOCE_STATIC_SCRATCH_BYTES, "header and library agree on the size");
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (taken on the first
// call there), or nullptr if the runtime cannot provide it.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

moce_status moce_forward(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                         const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  Shape sh;
  const moce_status st = check_forward(desc, x, s, w, gate, U, nU, y, &sh);
  if (st != MOCE_OK) return st;
  if (!ws || ws_bytes < ws_layout(sh).total) return MOCE_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return MOCE_ERR_ALIGN;
  return forward_launch(sh, x, s, w, gate, U, nU, y, ws, stream);
}

moce_status moce_forward_ex(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                            const moce_gate_params* gate, const int32_t* U, int32_t nU, const moce_epilogue* ep,
                            void* y, void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape sh;
  const moce_status st = check_forward(desc, x, s, w, gate, U, nU, y, &sh);
  if (st != MOCE_OK) return st;
  moce::Epi e{};
  if (ep) {
    if ((ep->scale == nullptr) != (ep->shift == nullptr)) return MOCE_ERR_NULL;
    e = moce::Epi{ep->scale, ep->shift, ep->relu != 0 ? 1 : 0};
  }
  if (!ws || ws_bytes < ws_layout(sh).total) return MOCE_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return MOCE_ERR_ALIGN;
  return forward_launch(sh, x, s, w, gate, U, nU, y, ws, stream, e);
}

moce_status moce_forward_static(const moce_desc* desc, const void* x, const int32_t* s, const float* w,
                                const moce_gate_params* gate, const int32_t* U, int32_t nU, void* y,
                                hipStream_t stream) {
  Shape sh;
  const moce_status st = check_forward(desc, x, s, w, gate, U, nU, y, &sh);
  if (st != MOCE_OK) return st;
  if (ws_layout(sh).total > kStaticScratchBytes) return MOCE_ERR_WORKSPACE;
  void* ws = scratch_on_current_device();
  if (!ws) return MOCE_ERR_DEVICE;
  // every region of the workspace is written before it is read (d by the
  // pooling, tau and the statistics or coefficients by the gate), so nothing
  // left by an earlier call is ever used
  return forward_launch(sh, x, s, w, gate, U, nU, y, ws, stream);
}

// ---- input-conditioned supports ------------------------------------------

namespace {

// Dynamic forward workspace: d [B][C], h [B][d], vT [d][C], S [B][R][k],
// W [B][R][k], U [B][C], nU [B], tau [B][R], alpha [B][R][k]; 256-byte
// aligned regions.
struct DynLayout {
  size_t d, h, vT, S, W, U, nU, tau, alpha, total;
};
DynLayout dyn_layout(const Shape& sh, int dd) {
  DynLayout l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += round_up(bytes);
    return at;
  };
  const size_t brk = (size_t)sh.B * sh.R * sh.k;
  l.d = take((size_t)sh.B * sh.C * sizeof(float));
  l.h = take((size_t)sh.B * dd * sizeof(float));
  l.vT = take((size_t)dd * sh.C * sizeof(float));
  l.S = take(brk * sizeof(int32_t));
  l.W = take(brk * sizeof(float));
  l.U = take((size_t)sh.B * sh.C * sizeof(int32_t));
  l.nU = take((size_t)sh.B * sizeof(int32_t));
  l.tau = take((size_t)sh.B * sh.R * sizeof(float));
  l.alpha = take(brk * sizeof(float));
  l.total = off;
  return l;
}

}  // namespace

size_t moce_forward_dynamic_workspace_bytes(const moce_desc* desc, int32_t d) {
  Shape sh;
  if (check_desc(desc, &sh) != MOCE_OK || d < 1 || !moce::dynamic_supported(sh, d)) return 0;
  return dyn_layout(sh, d).total;
}

moce_status moce_forward_dynamic(const moce_desc* desc, const void* x, const float* L, const moce_router* router,
                                 const moce_gate_params* gate, void* y, int32_t* S_out, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  st = check_gate(sh, gate);
  if (st != MOCE_OK) return st;
  if (!x || !y || !router) return MOCE_ERR_NULL;
  if (router->d < 1) return MOCE_ERR_SHAPE;
  if (sh.R > 0 && (!L || !router->Wh || !router->bh || !router->v || !router->q)) return MOCE_ERR_NULL;
  if (!moce::dynamic_supported(sh, router->d)) return MOCE_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y, 16)) return MOCE_ERR_ALIGN;
  const DynLayout l = dyn_layout(sh, router->d);
  if (!ws || ws_bytes < l.total) return MOCE_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return MOCE_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  int32_t* S = S_out ? S_out : reinterpret_cast<int32_t*>(base + l.S);
  return device_status(moce::launch_dynamic(
      sh, x, L, *router, *gate, y, reinterpret_cast<float*>(base + l.d), reinterpret_cast<float*>(base + l.h),
      reinterpret_cast<float*>(base + l.vT), S,
      reinterpret_cast<float*>(base + l.W), reinterpret_cast<int32_t*>(base + l.U),
      reinterpret_cast<int32_t*>(base + l.nU), reinterpret_cast<float*>(base + l.tau),
      reinterpret_cast<float*>(base + l.alpha), stream));
}

// ---- backward ----------------------------------------------------------------

namespace {

struct BwdLayout {
  size_t d, tau, stats, alpha, dal, S1, dtau, dg, dd, cnt, cur, off, inv, nU, dzg, part;
  size_t dxs_cnt, dxs_off, dxs_cur, dxs_w0, dxs_w1, dxs_coef, psum, total;
};
BwdLayout bwd_layout(const Shape& sh, int gate_kind) {
  BwdLayout l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += round_up(std::max<size_t>(bytes, 4));
    return at;
  };
  const size_t br = (size_t)sh.B * sh.R, brk = br * sh.k;
  l.d = take((size_t)sh.B * sh.C * sizeof(float));
  l.tau = take(br * sizeof(float));
  l.stats = take(3 * br * sizeof(float));
  int nbk = 0;
  int64_t nek = 0;
  moce::bwd_dx_sched_sizes(sh, &nbk, &nek);
  l.alpha = take(nbk > 0 ? 0 : brk * sizeof(float));
  int nsplit = 1, split_len = 0;
  moce::bwd_dalpha_splits(sh, &nsplit, &split_len);
  l.dal = take((size_t)nsplit * brk * sizeof(float));
  l.S1 = take(br * sizeof(float));
  l.dtau = take(br * sizeof(float));
  l.dg = take(br * sizeof(float));
  l.dd = take((size_t)sh.B * sh.C * sizeof(float));
  l.cnt = take((size_t)(sh.C + 1) * sizeof(int32_t));
  l.cur = take((size_t)sh.C * sizeof(int32_t));
  l.off = take((size_t)(sh.C + 1) * sizeof(int32_t));
  l.inv = take((size_t)sh.R * sh.k * sizeof(int32_t));
  l.nU = take(sizeof(int32_t));
  const bool mlp = gate_kind == MOCE_GATE_MLP_SIGMOID;
  l.dzg = take(mlp ? brk * sizeof(float) : 0);
  l.part = take(mlp ? moce::backward_mlp_parts(sh) * moce::backward_mlp_part_floats(sh) * sizeof(float) : 0);
  int nb = 0;
  int64_t ne = 0;
  moce::bwd_dx_sched_sizes(sh, &nb, &ne);
  l.dxs_cnt = take((size_t)nb * sizeof(int32_t));
  l.dxs_off = take((size_t)(nb + 1) * sizeof(int32_t));
  l.dxs_cur = take((size_t)nb * sizeof(int32_t));
  l.dxs_w0 = take((size_t)ne * sizeof(uint32_t));
  l.dxs_w1 = take((size_t)ne * sizeof(int32_t));
  l.dxs_coef = take((size_t)sh.B * ne * sizeof(uint32_t));
  int ng = 1, gs = 1;
  moce::backward_sum_groups(sh, &ng, &gs);
  l.psum = take((size_t)ng * (2 * (size_t)sh.R * sh.k + sh.R) * sizeof(float));
  l.total = off;
  return l;
}

}  // namespace

size_t moce_backward_workspace_bytes(const moce_desc* desc, int gate_kind) {
  Shape sh;
  if (check_desc(desc, &sh) != MOCE_OK) return 0;
  if (gate_kind != MOCE_GATE_SOFTPLUS_LINEAR && gate_kind != MOCE_GATE_MLP_SIGMOID) return 0;
  if (!moce::backward_supported(sh, gate_kind)) return 0;
  return bwd_layout(sh, gate_kind).total;
}

moce_status moce_backward(const moce_desc* desc, const void* x, const void* dy, const int32_t* s, const float* w,
                          const moce_gate_params* gate, void* dx, float* dw, const moce_gate_grads* grads,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape sh;
  moce_status st = check_desc(desc, &sh);
  if (st != MOCE_OK) return st;
  st = check_gate(sh, gate);
  if (st != MOCE_OK) return st;
  if (!x || !dy || !dx || !grads) return MOCE_ERR_NULL;
  const bool mlp = gate->kind == MOCE_GATE_MLP_SIGMOID;
  if (sh.R > 0) {
    if (!s || !w || !dw) return MOCE_ERR_NULL;
    if (mlp ? (!grads->dW1 || !grads->db1 || !grads->dw2 || !grads->db2) : (!grads->da || !grads->dc))
      return MOCE_ERR_NULL;
  }
  if (!moce::backward_supported(sh, gate->kind)) return MOCE_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(dy, 16) || !aligned(dx, 16)) return MOCE_ERR_ALIGN;
  const BwdLayout l = bwd_layout(sh, gate->kind);
  if (!ws || ws_bytes < l.total) return MOCE_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return MOCE_ERR_ALIGN;
  char* base = static_cast<char*>(ws);
  auto F = [&](size_t o) { return reinterpret_cast<float*>(base + o); };
  auto I = [&](size_t o) { return reinterpret_cast<int32_t*>(base + o); };
  const moce::BwdWs b{F(l.d),   F(l.tau),   F(l.stats), F(l.alpha), F(l.dal), F(l.S1),  F(l.dtau), F(l.dg),  F(l.dd),
                      I(l.cnt), I(l.cur),   I(l.off),   I(l.inv), I(l.nU),  F(l.dzg),  F(l.part),
                      I(l.dxs_cnt), I(l.dxs_off), I(l.dxs_cur),
                      reinterpret_cast<uint32_t*>(base + l.dxs_w0), I(l.dxs_w1),
                      reinterpret_cast<uint32_t*>(base + l.dxs_coef), F(l.psum)};
  return device_status(moce::launch_backward(sh, x, dy, s, w, *gate, dx, dw, *grads, b, stream));
}

size_t moce_logit_backward_workspace_bytes(int32_t R, int64_t C) {
  if (R < 1 || !moce::logit_backward_supported(C)) return 0;
  return round_up((2 * (size_t)R + (size_t)C + 3) * sizeof(float));
}

moce_status moce_logit_backward(int32_t R, int64_t C, int32_t k, const float* L, const int32_t* s, const float* dw,
                                float eps, float lambda, float* loss, float* dL, void* ws, size_t ws_bytes,
                                hipStream_t stream) {
  if (!L || !dL || !ws) return MOCE_ERR_NULL;
  if ((s == nullptr) != (dw == nullptr)) return MOCE_ERR_NULL;
  if (R < 1 || C < 1) return MOCE_ERR_SHAPE;
  if (dw && (k < 1 || (int64_t)k > C)) return MOCE_ERR_SHAPE;
  if (!std::isfinite(eps) || eps < 0.f || !std::isfinite(lambda)) return MOCE_ERR_SHAPE;
  if (!moce::logit_backward_supported(C)) return MOCE_ERR_UNSUPPORTED;
  if (ws_bytes < moce_logit_backward_workspace_bytes(R, C)) return MOCE_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return MOCE_ERR_ALIGN;
  return device_status(moce::launch_logit_backward(R, (int)C, k, L, s, dw, eps, lambda, loss, dL,
                                                   static_cast<float*>(ws), stream));
}

}  // extern "C"

// C ABI of the resonant mixing library: argument validation, workspace layout
// and kernel dispatch.  Declared in include/resonator.h.
#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdint>
#include <initializer_list>
#include <cstdio>
#include <mutex>
#include <string>

#include "../../include/resonator.h"
#include "common.h"
#include "kernels.h"

using namespace res;

namespace {

thread_local std::string g_err;
// Armed by resonator_set_kernel_timer for the next dominant-kernel launch.
thread_local hipEvent_t g_ev0 = nullptr, g_ev1 = nullptr;

void take_timer(hipEvent_t* e0, hipEvent_t* e1) {
  *e0 = g_ev0;
  *e1 = g_ev1;
  g_ev0 = g_ev1 = nullptr;
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(RES_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// compute units of the current device (256 if the query fails: only a launch
// shape depends on it)
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n < 1)
    return 256;
  return n;
}

}  // namespace

// Workspace of resonator_mix_fwd_noalloc: every GPU the library runs on holds
// its own copy until the process ends, zero at load like any device variable
// without an initialiser (a forward workspace must start zero-filled; each
// forward leaves it ready for the next).  Host code never passes this name to a
// kernel (on the host it is only a stand-in); it uses the device address that
// hipGetSymbolAddress gives for the current device.
static __device__ __align__(256) unsigned char scratch[RES_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[SCRATCH_MAX_DEVICES];  // device address of `scratch`, per device, taken once

// Device address of the static scratch on the device of `stream` (which must be
// the calling thread's current device), looked up on the first call per device.
int noalloc_scratch(void* stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (stream != nullptr) {
    hipDevice_t sdev = 0;
    if ((e = hipStreamGetDevice((hipStream_t)stream, &sdev)) != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if ((int)sdev != dev)
      return fail(RES_ERR_INVALID_ARG, "the stream belongs to device %d, the current device is %d", (int)sdev, dev);
  }
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES)
    return fail(RES_ERR_UNSUPPORTED, "device index %d beyond the %d the scratch table covers", dev,
                SCRATCH_MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
      return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr || ((uintptr_t)p % 256) != 0) return fail(RES_ERR_HIP, "scratch address unusable");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return RES_OK;
}

size_t elt_size(res_dtype_t t) { return t == RES_BF16 ? 2 : 4; }
bool dtype_ok(int t) { return t == RES_F32 || t == RES_BF16; }
bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Geometry of the tiled kernels for activations of type act (tile width depends
// on the element size: 128-byte rows).
Geometry make_geom(res_dtype_t act, int64_t B, int64_t L, int64_t D, int64_t M) {
  Geometry g;
  g.B = B;
  g.L = L;
  g.D = D;
  g.M = M;
  g.DW = act == RES_BF16 ? 64 : 32;
  g.NB = (int)((D + g.DW - 1) / g.DW);
  g.Dp = g.NB * g.DW;
  g.MG = (int)((M + MODES_PER_GROUP - 1) / MODES_PER_GROUP);
  g.Mp = MODES_PER_GROUP * g.MG;
  g.P = L > 0 ? (L + TILE_T - 1) / TILE_T : 0;
  g.last_len = L > 0 ? (int)(L - (g.P - 1) * TILE_T) : 0;
  return g;
}

// Workspace of the single-pass forward (M <= 8), byte offsets.  The first 256
// bytes are the header (status word first); the forward workspace must be zero
// before its first use and each call leaves it ready for the next.
struct StreamLayout {
  size_t hdr, chainw, agg, ring, total;
};
// The single-pass forward keeps per-chain counters in a fixed area of the
// workspace (every call resets the counters it used), ahead of the tagged
// states, so that one workspace serves calls of any shapes: a call's states
// never land on another call's counters.
constexpr int64_t STREAM_MAX_CHAINS = 1 << 16;
bool stream_forward(const Geometry& g) { return g.MG == 1 && g.B * g.NB <= STREAM_MAX_CHAINS; }

StreamLayout make_stream_layout(const Geometry& g) {
  StreamLayout w{};
  const size_t nchains = (size_t)g.B * g.NB, tiles = nchains * (size_t)g.P;
  // a tile's published end state: one 8-byte word per channel and state component
  const size_t state = (size_t)g.DW * 16 * sizeof(uint64_t);
  size_t off = 0;
  w.hdr = off;
  off += 256;
  w.chainw = off;
  off += (size_t)STREAM_MAX_CHAINS * 4 * sizeof(uint32_t);
  w.agg = off;
  off += align256(tiles * state);
  w.ring = off;
  off += align256((size_t)std::min(nchains, (size_t)STREAM_RING_CHAINS) * STREAM_RING * state);
  w.total = off;
  return w;
}

WsLayout make_layout(int op, res_dtype_t act, const Geometry& g) {
  WsLayout w{};
  size_t off = 0;
  (void)act;
  if (op == RES_OP_FWD) {
    if (stream_forward(g)) {
      w.total = make_stream_layout(g).total;
      return w;
    }
    off = 256;  // header (status word), as in the single-pass layout
  }
  const int nm = op == RES_OP_BWD ? bwd_mats(g.MG) : fwd_mats(g.MG);
  const size_t tiles_modes = (size_t)g.B * g.P * g.Dp * g.Mp;  // = tiles * DW * Mp
  w.tab = off;
  off += align256((size_t)g.Dp * nm * TAB_MAT_BYTES);
  w.scal = off;
  off += align256((size_t)g.Dp * g.Mp * sizeof(ModeScalars));
  w.carryc = off;
  off += align256((size_t)g.Dp * g.Mp * sizeof(ModeCarry));
  if (op == RES_OP_FWD || op == RES_OP_STATE_INIT) {
    // per tile [DW * Mp] float4 records: half-tile aggregates, then entry states
    w.agg = off;
    off += align256(tiles_modes * sizeof(float4));
    if (op == RES_OP_FWD) {
      w.carry = off;
      off += align256(tiles_modes * sizeof(float4));
    }
    w.alast = off;  // [B][Dp][Mp] state at t = L-1 from a zero start at the last tile
    off += align256((size_t)g.B * g.Dp * g.Mp * sizeof(float2));
  } else {
    // per segment (at most one per tile) records, partial sums, then q0
    w.agg = off;
    off += align256(tiles_modes * sizeof(float4));
    w.part = off;
    off += align256((size_t)g.B * g.P * g.Dp * (16 + 4 * g.Mp) * sizeof(float));
    w.q0 = off;
    off += align256((size_t)g.B * g.Dp * g.Mp * sizeof(float4));
  }
  w.total = off;
  return w;
}

int check_sizes(int64_t B, int64_t L, int64_t D, int64_t M, bool allow_l0) {
  if (B < 1 || D < 1) return fail(RES_ERR_INVALID_ARG, "B and D must be >= 1 (got B=%lld D=%lld)",
                                  (long long)B, (long long)D);
  if (L < (allow_l0 ? 0 : 1))
    return fail(RES_ERR_INVALID_ARG, "L must be >= %d (got %lld)", allow_l0 ? 0 : 1, (long long)L);
  if (M < 1 || M > RES_M_MAX)
    return fail(M < 1 ? RES_ERR_INVALID_ARG : RES_ERR_UNSUPPORTED,
                "M must be in [1, %d] (got %lld)", RES_M_MAX, (long long)M);
  if (D > (1 << 24) || B > (1LL << 31) || L > (1LL << 40))
    return fail(RES_ERR_UNSUPPORTED, "sizes beyond the supported range (B=%lld L=%lld D=%lld)",
                (long long)B, (long long)L, (long long)D);
  const int64_t tiles = B * ((L + TILE_T - 1) / TILE_T) * ((D + 31) / 32);
  if (tiles >= (1LL << 31))
    return fail(RES_ERR_UNSUPPORTED, "too many tiles for one launch (%lld)", (long long)tiles);
  return RES_OK;
}

int check_params(const float* gamma, const float* omega, const float* amp, const float* phase) {
  if (!gamma || !omega || !amp || !phase)
    return fail(RES_ERR_INVALID_ARG, "gamma, omega, amp and phase must be non-null");
  if (!aligned(gamma, 4) || !aligned(omega, 4) || !aligned(amp, 4) || !aligned(phase, 4))
    return fail(RES_ERR_MISALIGNED, "parameter arrays must be 4-byte aligned");
  return RES_OK;
}

bool overlap(const void* a, size_t an, const void* b, size_t bn) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + bn && y < x + an;
}

}  // namespace

extern "C" {

int resonator_version(void) { return 100; }

const char* resonator_last_error(void) { return g_err.c_str(); }

int resonator_set_kernel_timer(void* start_event, void* stop_event) {
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(RES_ERR_INVALID_ARG, "pass both events or neither");
  g_ev0 = (hipEvent_t)start_event;
  g_ev1 = (hipEvent_t)stop_event;
  return RES_OK;
}

size_t resonator_workspace_bytes(int op, res_dtype_t act_dt, int64_t B, int64_t L, int64_t D,
                                 int64_t M) {
  if (op != RES_OP_FWD && op != RES_OP_BWD && op != RES_OP_STATE_INIT) return 0;
  if (!dtype_ok(act_dt)) return 0;
  if (B < 1 || D < 1 || M < 1 || M > RES_M_MAX || L < (op == RES_OP_STATE_INIT ? 0 : 1)) return 0;
  if (L == 0) return 0;
  return make_layout(op, act_dt, make_geom(act_dt, B, L, D, M)).total;
}

}  // extern "C"

namespace {

// Validation and dispatch of the forward; noalloc: the allocation-free entry
// point (ws and ws_bytes ignored, the workspace is the device's static scratch).
int mix_fwd_impl(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B, int64_t L, int64_t D,
                 int64_t M, const float* gamma, const float* omega, const float* amp, const float* phase,
                 const float* h0, float* h_out, void* ws, size_t ws_bytes, void* stream, bool noalloc) {
  int rc = check_sizes(B, L, D, M, false);
  if (rc) return rc;
  if (!dtype_ok(x_dt) || !dtype_ok(y_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (x_dt == RES_F32 && y_dt == RES_BF16)
    return fail(RES_ERR_UNSUPPORTED, "dtype pair f32 -> bf16 is not supported");
  if (!x || !y) return fail(RES_ERR_INVALID_ARG, "x and y must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  if (!aligned(x, elt_size(x_dt)) || !aligned(y, elt_size(y_dt)) || (h0 && !aligned(h0, 4)) ||
      (h_out && !aligned(h_out, 4)))
    return fail(RES_ERR_MISALIGNED, "activation/state pointers must be aligned to their element");
  const size_t n = (size_t)(B * L * D);
  if (overlap(x, n * elt_size(x_dt), y, n * elt_size(y_dt)))
    return fail(RES_ERR_INVALID_ARG, "y must not overlap x");
  const Geometry g = make_geom(x_dt, B, L, D, M);
  const WsLayout w = make_layout(RES_OP_FWD, x_dt, g);
  if (noalloc) {
    if (w.total > (size_t)RES_NOALLOC_SCRATCH_BYTES)
      return fail(RES_ERR_WORKSPACE,
                  "sizes need %zu bytes of workspace, more than the %zu-byte static scratch of "
                  "resonator_mix_fwd_noalloc; call resonator_mix_fwd with a workspace",
                  w.total, (size_t)RES_NOALLOC_SCRATCH_BYTES);
    if ((rc = noalloc_scratch(stream, &ws))) return rc;
    ws_bytes = (size_t)RES_NOALLOC_SCRATCH_BYTES;
  }
  if (!ws || ws_bytes < w.total)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", w.total, ws_bytes);
  if (!aligned(ws, 256)) return fail(RES_ERR_MISALIGNED, "workspace must be 256-byte aligned");

  hipStream_t st = (hipStream_t)stream;
  char* base = (char*)ws;
  // 16-byte row segments: both activation pointers 16-byte aligned, rows a multiple of 16 bytes
  const int fast_io = aligned(x, 16) && aligned(y, 16) && (D * elt_size(x_dt)) % 16 == 0 &&
                      (D * elt_size(y_dt)) % 16 == 0;
  hipEvent_t ev0, ev1;
  take_timer(&ev0, &ev1);
  hipError_t e;
  if (stream_forward(g)) {  // single-pass forward
    const StreamLayout sl = make_stream_layout(g);
    int dev = 0, ncu = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return hip_fail(e, "hipGetDevice");
    if ((e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return hip_fail(e, "device attribute");
    StreamArgs a{};
    a.x = x;
    a.y = y;
    a.B = B;
    a.L = L;
    a.D = (int)D;
    a.M = (int)M;
    a.NB = g.NB;
    a.nchains = (int)(B * g.NB);
    a.P = g.P;
    a.last_len = g.last_len;
    a.fast_io = fast_io;
    a.gamma = gamma;
    a.omega = omega;
    a.amp = amp;
    a.phase = phase;
    a.h0 = h0;
    a.h_out = h_out;
    a.hdr = (uint32_t*)(base + sl.hdr);
    a.chainw = (uint32_t*)(base + sl.chainw);
    a.agg = (uint64_t*)(base + sl.agg);
    a.ring = B * g.NB <= STREAM_RING_CHAINS ? (uint64_t*)(base + sl.ring) : nullptr;
    const int grid = fwd_stream_grid(B * g.NB, g.P, ncu > 0 ? ncu : 256);
    if (x_dt == RES_F32)
      e = launch_fwd_stream<float, float>(a, grid, st, ev0, ev1);
    else if (y_dt == RES_BF16)
      e = launch_fwd_stream<bf16_t, bf16_t>(a, grid, st, ev0, ev1);
    else
      e = launch_fwd_stream<bf16_t, float>(a, grid, st, ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "forward launch");
    return RES_OK;
  }
  ModeScalars* scal = (ModeScalars*)(base + w.scal);
  ModeCarry* cc = (ModeCarry*)(base + w.carryc);
  e = x_dt == RES_BF16
          ? launch_prep<bf16_t>(g, gamma, omega, amp, phase, false, base + w.tab, scal, cc, st)
          : launch_prep<float>(g, gamma, omega, amp, phase, false, base + w.tab, scal, cc, st);
  if (e != hipSuccess) return hip_fail(e, "prep launch");
  FwdArgs a{};
  a.x = x;
  a.y = y;
  a.B = B;
  a.L = L;
  a.D = (int)D;
  a.M = (int)M;
  a.NB = g.NB;
  a.Dp = g.Dp;
  a.Mp = g.Mp;
  a.P = g.P;
  a.last_len = g.last_len;
  a.fast_io = fast_io;
  a.tab = base + w.tab;
  a.scal = scal;
  a.cc = cc;
  a.h0 = h0;
  a.h_out = h_out;
  a.agg = base + w.agg;
  a.car = base + w.carry;
  a.alast = (float2*)(base + w.alast);
  e = x_dt == RES_F32 ? launch_fwd_agg<float>(g, a, st) : launch_fwd_agg<bf16_t>(g, a, st);
  if (e != hipSuccess) return hip_fail(e, "aggregate launch");
  if ((e = launch_fwd_carry(g, a, st)) != hipSuccess) return hip_fail(e, "carry launch");
  if (x_dt == RES_F32)
    e = launch_fwd_apply<float, float>(g, a, st, ev0, ev1);
  else if (y_dt == RES_BF16)
    e = launch_fwd_apply<bf16_t, bf16_t>(g, a, st, ev0, ev1);
  else
    e = launch_fwd_apply<bf16_t, float>(g, a, st, ev0, ev1);
  if (e != hipSuccess) return hip_fail(e, "apply launch");
  return RES_OK;
}

}  // namespace

extern "C" {

int resonator_mix_fwd(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B,
                      int64_t L, int64_t D, int64_t M, const float* gamma, const float* omega,
                      const float* amp, const float* phase, const float* h0, float* h_out,
                      void* ws, size_t ws_bytes, void* stream) {
  return mix_fwd_impl(x, x_dt, y, y_dt, B, L, D, M, gamma, omega, amp, phase, h0, h_out, ws, ws_bytes, stream,
                      false);
}

int resonator_mix_fwd_noalloc(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B, int64_t L,
                              int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                              const float* phase, const float* h0, float* h_out, void* stream) {
  return mix_fwd_impl(x, x_dt, y, y_dt, B, L, D, M, gamma, omega, amp, phase, h0, h_out, nullptr, 0, stream,
                      true);
}

size_t resonator_mix_fwd_noalloc_max_bytes(void) { return (size_t)RES_NOALLOC_SCRATCH_BYTES; }

int resonator_fwd_status(void* ws, uint32_t* status, void* stream) {
  if (!ws || !status) return fail(RES_ERR_INVALID_ARG, "ws and status must be non-null");
  if (!aligned(ws, 256)) return fail(RES_ERR_MISALIGNED, "workspace must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if ((e = hipMemcpyAsync(status, ws, sizeof(uint32_t), hipMemcpyDeviceToHost, st)) != hipSuccess)
    return hip_fail(e, "status copy");
  if ((e = hipMemsetAsync(ws, 0, sizeof(uint32_t), st)) != hipSuccess) return hip_fail(e, "status clear");
  if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_fail(e, "status synchronize");
  return RES_OK;
}

int resonator_fwd_status_noalloc(uint32_t* status, void* stream) {
  void* ws = nullptr;
  const int rc = noalloc_scratch(stream, &ws);
  if (rc) return rc;
  return resonator_fwd_status(ws, status, stream);
}

int resonator_state_init(const void* x_prompt, res_dtype_t x_dt, int64_t B, int64_t L_prompt,
                         int64_t D, int64_t M, const float* gamma, const float* omega,
                         const float* amp, const float* phase, float* state_out, void* ws,
                         size_t ws_bytes, void* stream) {
  int rc = check_sizes(B, L_prompt, D, M, true);
  if (rc) return rc;
  if (!dtype_ok(x_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!state_out) return fail(RES_ERR_INVALID_ARG, "state_out must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  if (!aligned(state_out, 4)) return fail(RES_ERR_MISALIGNED, "state_out must be 4-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  if (L_prompt == 0) {
    const hipError_t e = launch_fill_zero(state_out, B * D * M * 2, st);
    return e == hipSuccess ? RES_OK : hip_fail(e, "fill launch");
  }
  if (!x_prompt) return fail(RES_ERR_INVALID_ARG, "x_prompt must be non-null when L_prompt > 0");
  if (!aligned(x_prompt, elt_size(x_dt))) return fail(RES_ERR_MISALIGNED, "x_prompt misaligned");
  const Geometry g = make_geom(x_dt, B, L_prompt, D, M);
  const WsLayout w = make_layout(RES_OP_STATE_INIT, x_dt, g);
  if (!ws || ws_bytes < w.total)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", w.total, ws_bytes);
  if (!aligned(ws, 256)) return fail(RES_ERR_MISALIGNED, "workspace must be 256-byte aligned");
  char* base = (char*)ws;
  ModeScalars* scal = (ModeScalars*)(base + w.scal);
  ModeCarry* cc = (ModeCarry*)(base + w.carryc);
  hipError_t e =
      x_dt == RES_BF16
          ? launch_prep<bf16_t>(g, gamma, omega, amp, phase, false, base + w.tab, scal, cc, st)
          : launch_prep<float>(g, gamma, omega, amp, phase, false, base + w.tab, scal, cc, st);
  if (e != hipSuccess) return hip_fail(e, "prep launch");
  FwdArgs a{};
  a.x = x_prompt;
  a.y = nullptr;
  a.B = B;
  a.L = L_prompt;
  a.D = (int)D;
  a.M = (int)M;
  a.NB = g.NB;
  a.Dp = g.Dp;
  a.Mp = g.Mp;
  a.P = g.P;
  a.last_len = g.last_len;
  a.fast_io = aligned(x_prompt, 16) && (D * elt_size(x_dt)) % 16 == 0;
  a.tab = base + w.tab;
  a.scal = scal;
  a.cc = cc;
  a.h_out = state_out;
  a.agg = base + w.agg;
  a.car = nullptr;
  a.alast = (float2*)(base + w.alast);
  e = x_dt == RES_F32 ? launch_fwd_agg<float>(g, a, st) : launch_fwd_agg<bf16_t>(g, a, st);
  if (e != hipSuccess) return hip_fail(e, "aggregate launch");
  if ((e = launch_fwd_carry(g, a, st)) != hipSuccess) return hip_fail(e, "carry launch");
  return RES_OK;
}

int resonator_mix_bwd(const void* x, const void* dy, res_dtype_t act_dt, void* dx, int64_t B,
                      int64_t L, int64_t D, int64_t M, const float* gamma, const float* omega,
                      const float* amp, const float* phase, const float* h0, float* dgamma,
                      float* domega, float* damp, float* dphase, float* dh0, void* ws,
                      size_t ws_bytes, void* stream) {
  int rc = check_sizes(B, L, D, M, false);
  if (rc) return rc;
  if (!dtype_ok(act_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!x || !dy || !dx) return fail(RES_ERR_INVALID_ARG, "x, dy and dx must be non-null");
  if (!dgamma || !domega || !damp || !dphase)
    return fail(RES_ERR_INVALID_ARG, "dgamma, domega, damp and dphase must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  const size_t es = elt_size(act_dt);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(dx, es) || (h0 && !aligned(h0, 4)) ||
      (dh0 && !aligned(dh0, 4)) || !aligned(dgamma, 4) || !aligned(domega, 4) ||
      !aligned(damp, 4) || !aligned(dphase, 4))
    return fail(RES_ERR_MISALIGNED, "pointers must be aligned to their element");
  const size_t n = (size_t)(B * L * D) * es;
  if (overlap(dx, n, x, n) || overlap(dx, n, dy, n))
    return fail(RES_ERR_INVALID_ARG, "dx must not overlap x or dy");
  const Geometry g = make_geom(act_dt, B, L, D, M);
  const WsLayout w = make_layout(RES_OP_BWD, act_dt, g);
  if (!ws || ws_bytes < w.total)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", w.total, ws_bytes);
  if (!aligned(ws, 256)) return fail(RES_ERR_MISALIGNED, "workspace must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  char* base = (char*)ws;
  ModeScalars* scal = (ModeScalars*)(base + w.scal);
  ModeCarry* cc = (ModeCarry*)(base + w.carryc);
  hipError_t e =
      act_dt == RES_BF16
          ? launch_prep<bf16_t>(g, gamma, omega, amp, phase, true, base + w.tab, scal, cc, st)
          : launch_prep<float>(g, gamma, omega, amp, phase, true, base + w.tab, scal, cc, st);
  if (e != hipSuccess) return hip_fail(e, "prep launch");
  int dev = 0, ncu = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return hip_fail(e, "hipGetDevice");
  if ((e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
    return hip_fail(e, "device attribute");
  BwdArgs a{};
  a.x = x;
  a.dy = dy;
  a.dx = dx;
  a.B = B;
  a.L = L;
  a.D = (int)D;
  a.M = (int)M;
  const int dwb = bwd_block_channels((int)es);
  a.NB = (int)((D + dwb - 1) / dwb);
  a.Dp = g.Dp;
  a.Mp = g.Mp;
  a.P = g.P;
  a.nseg = bwd_segments(B * a.NB, g.P, ncu);
  a.S = (g.P + a.nseg - 1) / a.nseg;
  a.nseg = (int)((g.P + a.S - 1) / a.S);
  // float32 drives, one mode group and an even number of tiles per segment:
  // records per half segment, so that the record pass runs two work-groups (of
  // four waves) per compute unit
  a.sf = (es == 4 && a.S % 2 == 0 && g.Mp == MODES_PER_GROUP) ? 2 : 1;
  a.Ss = a.S / a.sf;
  a.nss = (int)((g.P + a.Ss - 1) / a.Ss);
  a.fast_io = aligned(x, 16) && aligned(dy, 16) && aligned(dx, 16) && (D * (int64_t)es) % 16 == 0;
  a.tab = base + w.tab;
  a.scal = scal;
  a.cc = cc;
  a.agg = (float4*)(base + w.agg);
  a.part = (float*)(base + w.part);
  a.q0 = (float4*)(base + w.q0);
  hipEvent_t ev0, ev1;
  take_timer(&ev0, &ev1);
  e = act_dt == RES_BF16 ? launch_bwd<bf16_t>(a, st, ev0, ev1) : launch_bwd<float>(a, st, ev0, ev1);
  if (e != hipSuccess) return hip_fail(e, "bwd launch");
  if ((e = launch_bwd_reduce(g, a.nseg, a.part, a.q0, cc, h0, dgamma, domega, damp, dphase, dh0, st)) !=
      hipSuccess)
    return hip_fail(e, "bwd reduce launch");
  return RES_OK;
}

int resonator_decode_step(const void* x_t, res_dtype_t x_dt, void* y_t, res_dtype_t y_dt,
                          int64_t B, int64_t D, int64_t M, const float* gamma, const float* omega,
                          const float* amp, const float* phase, float* state, void* stream) {
  int rc = check_sizes(B, 1, D, M, false);
  if (rc) return rc;
  if (!dtype_ok(x_dt) || !dtype_ok(y_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (x_dt == RES_F32 && y_dt == RES_BF16)
    return fail(RES_ERR_UNSUPPORTED, "dtype pair f32 -> bf16 is not supported");
  if (!x_t || !y_t || !state) return fail(RES_ERR_INVALID_ARG, "x_t, y_t and state must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  if (!aligned(x_t, elt_size(x_dt)) || !aligned(y_t, elt_size(y_dt)) || !aligned(state, 8))
    return fail(RES_ERR_MISALIGNED, "x_t/y_t aligned to their element, state to 8 bytes");
  const size_t n = (size_t)(B * D);
  if (overlap(y_t, n * elt_size(y_dt), x_t, n * elt_size(x_dt)) ||
      overlap(y_t, n * elt_size(y_dt), state, n * M * 8))
    return fail(RES_ERR_INVALID_ARG, "y_t must not overlap x_t or state");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (x_dt == RES_F32)
    e = launch_decode<float, float>(B, D, M, x_t, y_t, gamma, omega, amp, phase, state, st);
  else if (y_dt == RES_BF16)
    e = launch_decode<bf16_t, bf16_t>(B, D, M, x_t, y_t, gamma, omega, amp, phase, state, st);
  else
    e = launch_decode<bf16_t, float>(B, D, M, x_t, y_t, gamma, omega, amp, phase, state, st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "decode launch");
}

int resonator_decode_constants(int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                               const float* phase, float* tab, void* stream) {
  int rc = check_sizes(1, 1, D, M, false);
  if (rc) return rc;
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  if (!tab) return fail(RES_ERR_INVALID_ARG, "tab must be non-null");
  if (!aligned(tab, 8)) return fail(RES_ERR_MISALIGNED, "tab must be 8-byte aligned");
  if (overlap(tab, (size_t)(D * M) * 24, gamma, (size_t)(D * M) * 4) ||
      overlap(tab, (size_t)(D * M) * 24, omega, (size_t)(D * M) * 4) ||
      overlap(tab, (size_t)(D * M) * 24, amp, (size_t)(D * M) * 4) ||
      overlap(tab, (size_t)(D * M) * 24, phase, (size_t)(D * M) * 4))
    return fail(RES_ERR_INVALID_ARG, "tab must not overlap the parameters");
  const hipError_t e = launch_decode_consts(D, M, gamma, omega, amp, phase, tab, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "decode constants launch");
}

int resonator_decode_step_tab(const void* x_t, res_dtype_t x_dt, void* y_t, res_dtype_t y_dt, int64_t B,
                              int64_t D, int64_t M, const float* tab, float* state, void* stream) {
  int rc = check_sizes(B, 1, D, M, false);
  if (rc) return rc;
  if (!dtype_ok(x_dt) || !dtype_ok(y_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (x_dt == RES_F32 && y_dt == RES_BF16)
    return fail(RES_ERR_UNSUPPORTED, "dtype pair f32 -> bf16 is not supported");
  if (!x_t || !y_t || !state || !tab) return fail(RES_ERR_INVALID_ARG, "x_t, y_t, tab and state must be non-null");
  if (!aligned(x_t, elt_size(x_dt)) || !aligned(y_t, elt_size(y_dt)) || !aligned(state, 8) || !aligned(tab, 8))
    return fail(RES_ERR_MISALIGNED, "x_t/y_t aligned to their element, state and tab to 8 bytes");
  const size_t n = (size_t)(B * D);
  if (overlap(y_t, n * elt_size(y_dt), x_t, n * elt_size(x_dt)) ||
      overlap(y_t, n * elt_size(y_dt), state, n * M * 8) || overlap(y_t, n * elt_size(y_dt), tab, (size_t)(D * M) * 24) ||
      overlap(state, n * M * 8, tab, (size_t)(D * M) * 24))
    return fail(RES_ERR_INVALID_ARG, "y_t must not overlap x_t, state or tab, nor state tab");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (x_dt == RES_F32)
    e = launch_decode_tab<float, float>(B, D, M, x_t, y_t, tab, state, st);
  else if (y_dt == RES_BF16)
    e = launch_decode_tab<bf16_t, bf16_t>(B, D, M, x_t, y_t, tab, state, st);
  else
    e = launch_decode_tab<bf16_t, float>(B, D, M, x_t, y_t, tab, state, st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "decode launch");
}

int resonator_decode_steps(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B, int64_t N,
                           int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                           const float* phase, float* state, void* stream) {
  int rc = check_sizes(B, N, D, M, false);
  if (rc) return rc;
  if (B > 4 * 65535LL) return fail(RES_ERR_UNSUPPORTED, "B must be <= %lld for this launch (got %lld)",
                                   4 * 65535LL, (long long)B);
  if (!dtype_ok(x_dt) || !dtype_ok(y_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (x_dt == RES_F32 && y_dt == RES_BF16)
    return fail(RES_ERR_UNSUPPORTED, "dtype pair f32 -> bf16 is not supported");
  if (!x || !y || !state) return fail(RES_ERR_INVALID_ARG, "x, y and state must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  if (!aligned(x, elt_size(x_dt)) || !aligned(y, elt_size(y_dt)) || !aligned(state, 8))
    return fail(RES_ERR_MISALIGNED, "x/y aligned to their element, state to 8 bytes");
  const size_t n = (size_t)(B * N * D);
  if (overlap(y, n * elt_size(y_dt), x, n * elt_size(x_dt)) ||
      overlap(y, n * elt_size(y_dt), state, (size_t)(B * D * M) * 8))
    return fail(RES_ERR_INVALID_ARG, "y must not overlap x or state");
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  if (x_dt == RES_F32)
    e = launch_decode_steps<float, float>(B, N, D, M, x, y, gamma, omega, amp, phase, state, st);
  else if (y_dt == RES_BF16)
    e = launch_decode_steps<bf16_t, bf16_t>(B, N, D, M, x, y, gamma, omega, amp, phase, state, st);
  else
    e = launch_decode_steps<bf16_t, float>(B, N, D, M, x, y, gamma, omega, amp, phase, state, st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "decode steps launch");
}

// ---------------------------------------------------------------------------
// Grouped linear projection (Sec. 3.1, 3.4)
// ---------------------------------------------------------------------------
int resonator_grouped_linear(const void* x, const void* W, res_dtype_t dt, void* y, int64_t N, int64_t d_in,
                             int64_t d_out, int64_t G, void* stream) {
  if (N < 1 || d_in < 1 || d_out < 1 || G < 1)
    return fail(RES_ERR_INVALID_ARG, "N, d_in, d_out and G must be >= 1");
  if (d_in % G || d_out % G)
    return fail(RES_ERR_INVALID_ARG, "d_in (%lld) and d_out (%lld) must be multiples of G (%lld)", (long long)d_in,
                (long long)d_out, (long long)G);
  if (N > INT32_MAX || d_in > INT32_MAX || d_out > INT32_MAX)
    return fail(RES_ERR_UNSUPPORTED, "N, d_in and d_out must be below 2^31");
  if (!dtype_ok(dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!x || !W || !y) return fail(RES_ERR_INVALID_ARG, "x, W and y must be non-null");
  const size_t es = elt_size(dt);
  if (!aligned(x, es) || !aligned(W, es) || !aligned(y, es))
    return fail(RES_ERR_MISALIGNED, "x, W and y must be aligned to their element");
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * es;
  if (overlap(y, ny, x, nx) || overlap(y, ny, W, nw)) return fail(RES_ERR_INVALID_ARG, "y must not overlap x or W");
  const bool bf = dt == RES_BF16;
  if (grouped_proj_supported(x, W, nullptr, y, nullptr, d_in, d_out, G, bf)) {
    const hipError_t e = launch_grouped_proj(x, W, nullptr, y, nullptr, N, d_in, d_out, G, bf, device_cus(),
                                             (hipStream_t)stream);
    return e == hipSuccess ? RES_OK : hip_fail(e, "grouped projection launch");
  }
  const char* err = launch_grouped_linear(x, W, y, N, d_in, d_out, G, bf, (hipStream_t)stream);
  if (err) return fail(RES_ERR_HIP, "grouped linear: %s", err);
  return RES_OK;
}

int resonator_grouped_linear2(const void* x, const void* W0, const void* W1, res_dtype_t dt, void* y0, void* y1,
                              int64_t N, int64_t d_in, int64_t d_out, int64_t G, void* stream) {
  if (N < 1 || d_in < 1 || d_out < 1 || G < 1)
    return fail(RES_ERR_INVALID_ARG, "N, d_in, d_out and G must be >= 1");
  if (d_in % G || d_out % G)
    return fail(RES_ERR_INVALID_ARG, "d_in (%lld) and d_out (%lld) must be multiples of G (%lld)", (long long)d_in,
                (long long)d_out, (long long)G);
  if (N > INT32_MAX || d_in > INT32_MAX || d_out > INT32_MAX)
    return fail(RES_ERR_UNSUPPORTED, "N, d_in and d_out must be below 2^31");
  if (!dtype_ok(dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!x || !W0 || !W1 || !y0 || !y1) return fail(RES_ERR_INVALID_ARG, "x, W0, W1, y0 and y1 must be non-null");
  const size_t es = elt_size(dt);
  if (!aligned(x, es) || !aligned(W0, es) || !aligned(W1, es) || !aligned(y0, es) || !aligned(y1, es))
    return fail(RES_ERR_MISALIGNED, "x, W0, W1, y0 and y1 must be aligned to their element");
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * es;
  if (overlap(y0, ny, x, nx) || overlap(y0, ny, W0, nw) || overlap(y0, ny, W1, nw) || overlap(y1, ny, x, nx) ||
      overlap(y1, ny, W0, nw) || overlap(y1, ny, W1, nw) || overlap(y0, ny, y1, ny))
    return fail(RES_ERR_INVALID_ARG, "y0 and y1 must overlap neither each other, x, W0 nor W1");
  const bool bf = dt == RES_BF16;
  if (grouped_proj_supported(x, W0, W1, y0, y1, d_in, d_out, G, bf)) {
    const hipError_t e = launch_grouped_proj(x, W0, W1, y0, y1, N, d_in, d_out, G, bf, device_cus(),
                                             (hipStream_t)stream);
    return e == hipSuccess ? RES_OK : hip_fail(e, "grouped projection launch");
  }
  const char* err = launch_grouped_linear(x, W0, y0, N, d_in, d_out, G, bf, (hipStream_t)stream);
  if (!err) err = launch_grouped_linear(x, W1, y1, N, d_in, d_out, G, bf, (hipStream_t)stream);
  if (err) return fail(RES_ERR_HIP, "grouped linear: %s", err);
  return RES_OK;
}

static int gl_check(int64_t N, int64_t d_in, int64_t d_out, int64_t G, res_dtype_t dt) {
  if (N < 1 || d_in < 1 || d_out < 1 || G < 1)
    return fail(RES_ERR_INVALID_ARG, "N, d_in, d_out and G must be >= 1");
  if (d_in % G || d_out % G)
    return fail(RES_ERR_INVALID_ARG, "d_in (%lld) and d_out (%lld) must be multiples of G (%lld)", (long long)d_in,
                (long long)d_out, (long long)G);
  if (N > INT32_MAX || d_in > INT32_MAX || d_out > INT32_MAX)
    return fail(RES_ERR_UNSUPPORTED, "N, d_in and d_out must be below 2^31");
  if (!dtype_ok(dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  return RES_OK;
}

int resonator_grouped_linear_bwd_data_sum(int n, const void* const* dy, const void* const* W, res_dtype_t dt,
                                          void* dx, int64_t N, int64_t d_in, int64_t d_out, int64_t G,
                                          int accumulate, void* stream) {
  int rc = gl_check(N, d_in, d_out, G, dt);
  if (rc) return rc;
  if (n < 1 || n > 3) return fail(RES_ERR_INVALID_ARG, "n must be 1, 2 or 3 (got %d)", n);
  if (!dy || !W || !dx) return fail(RES_ERR_INVALID_ARG, "dy, W and dx must be non-null");
  const size_t es = elt_size(dt);
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * es;
  if (!aligned(dx, es)) return fail(RES_ERR_MISALIGNED, "dx must be aligned to its element");
  for (int i = 0; i < n; ++i) {
    if (!dy[i] || !W[i]) return fail(RES_ERR_INVALID_ARG, "dy[%d] and W[%d] must be non-null", i, i);
    if (!aligned(dy[i], es) || !aligned(W[i], es))
      return fail(RES_ERR_MISALIGNED, "dy[%d] and W[%d] must be aligned to their element", i, i);
    if (overlap(dx, nx, dy[i], ny) || overlap(dx, nx, W[i], nw))
      return fail(RES_ERR_INVALID_ARG, "dx must not overlap dy[%d] or W[%d]", i, i);
  }
  const bool bf = dt == RES_BF16;
  if (grouped_dgrad_supported(n, dy, W, dx, d_in, d_out, G, bf)) {
    const hipError_t e = launch_grouped_dgrad(n, dy, W, dx, N, d_in, d_out, G, bf, accumulate != 0, device_cus(),
                                              (hipStream_t)stream);
    return e == hipSuccess ? RES_OK : hip_fail(e, "grouped data-gradient launch");
  }
  for (int i = 0; i < n; ++i) {
    const char* err = launch_grouped_linear_bwd_data(dy[i], W[i], dx, N, d_in, d_out, G, bf,
                                                     accumulate != 0 || i > 0, (hipStream_t)stream);
    if (err) return fail(RES_ERR_HIP, "grouped linear backward (data): %s", err);
  }
  return RES_OK;
}

int resonator_grouped_linear_bwd_data(const void* dy, const void* W, res_dtype_t dt, void* dx, int64_t N,
                                      int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* stream) {
  const void* dys[1] = {dy};
  const void* Ws[1] = {W};
  if (!dy || !W) return fail(RES_ERR_INVALID_ARG, "dy, W and dx must be non-null");
  return resonator_grouped_linear_bwd_data_sum(1, dys, Ws, dt, dx, N, d_in, d_out, G, accumulate, stream);
}

size_t resonator_grouped_linear_bwd_weight_sum_workspace_bytes(int n, int nout, int64_t N, int64_t d_in,
                                                                int64_t d_out, int64_t G, res_dtype_t dt) {
  if (N < 1 || d_in < 1 || d_out < 1 || G < 1) return 0;
  const int nb = grouped_wgrad_blocks(n, nout, d_in, d_out, G, dt == RES_BF16);
  return nb ? (size_t)grouped_wgrad_grid(N, n) * (size_t)nb * 1024 : 0;
}

int resonator_grouped_linear_bwd_weight_sum(int n, const void* x, const void* const* dy, const int* out,
                                            res_dtype_t dt, float* dW0, float* dW1, int64_t N, int64_t d_in,
                                            int64_t d_out, int64_t G, int accumulate, void* ws, size_t ws_bytes,
                                            void* stream) {
  int rc = gl_check(N, d_in, d_out, G, dt);
  if (rc) return rc;
  if (n < 1 || n > 3) return fail(RES_ERR_INVALID_ARG, "n must be 1, 2 or 3 (got %d)", n);
  if (!x || !dy || !out || !dW0) return fail(RES_ERR_INVALID_ARG, "x, dy, out and dW0 must be non-null");
  int nout = 1, used0 = 0;
  for (int i = 0; i < n; ++i) {
    if (out[i] != 0 && out[i] != 1) return fail(RES_ERR_INVALID_ARG, "out[%d] must be 0 or 1", i);
    if (!dy[i]) return fail(RES_ERR_INVALID_ARG, "dy[%d] must be non-null", i);
    if (out[i] == 1) nout = 2;
    else used0 = 1;
  }
  if (!used0) return fail(RES_ERR_INVALID_ARG, "at least one gradient must go to dW0");
  if (nout == 2 && !dW1) return fail(RES_ERR_INVALID_ARG, "dW1 must be non-null when out names weight 1");
  const size_t es = elt_size(dt);
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * 4;
  if (!aligned(x, es) || !aligned(dW0, 4) || (nout == 2 && !aligned(dW1, 4)))
    return fail(RES_ERR_MISALIGNED, "x aligned to its element, dW0 and dW1 to 4 bytes");
  float* const dWs[2] = {dW0, nout == 2 ? dW1 : nullptr};
  for (int m = 0; m < nout; ++m) {
    if (overlap(dWs[m], nw, x, nx)) return fail(RES_ERR_INVALID_ARG, "dW%d must not overlap x", m);
    if (ws && ws_bytes && overlap(dWs[m], nw, ws, ws_bytes))
      return fail(RES_ERR_INVALID_ARG, "dW%d must not overlap the workspace", m);
  }
  if (nout == 2 && overlap(dW0, nw, dW1, nw)) return fail(RES_ERR_INVALID_ARG, "dW0 and dW1 must not overlap");
  for (int i = 0; i < n; ++i) {
    if (!aligned(dy[i], es)) return fail(RES_ERR_MISALIGNED, "dy[%d] must be aligned to its element", i);
    for (int m = 0; m < nout; ++m)
      if (overlap(dWs[m], nw, dy[i], ny)) return fail(RES_ERR_INVALID_ARG, "dW%d must not overlap dy[%d]", m, i);
    if (ws && ws_bytes && overlap(ws, ws_bytes, dy[i], ny))
      return fail(RES_ERR_INVALID_ARG, "the workspace must not overlap dy[%d]", i);
  }
  if (ws && ws_bytes && overlap(ws, ws_bytes, x, nx)) return fail(RES_ERR_INVALID_ARG, "the workspace must not overlap x");
  const bool bf = dt == RES_BF16;
  bool al16 = ((uintptr_t)x & 15) == 0;
  for (int i = 0; i < n; ++i) al16 = al16 && ((uintptr_t)dy[i] & 15) == 0;
  const size_t need = resonator_grouped_linear_bwd_weight_sum_workspace_bytes(n, nout, N, d_in, d_out, G, dt);
  if (need > 0 && al16) {
    if (!ws || ws_bytes < need || !aligned(ws, 16))
      return fail(RES_ERR_INVALID_ARG, "workspace of %zu bytes (16-byte aligned) needed, got %zu", need, ws_bytes);
    const hipError_t e = launch_grouped_wgrad(n, x, dy, out, dW0, dW1, N, d_in, d_out, G, accumulate != 0,
                                              static_cast<float*>(ws), (hipStream_t)stream);
    return e == hipSuccess ? RES_OK : hip_fail(e, "grouped weight-gradient launch");
  }
  int first[2] = {1, 1};
  for (int i = 0; i < n; ++i) {
    const int m = out[i];
    const char* err = launch_grouped_linear_bwd_weight(x, dy[i], dWs[m], N, d_in, d_out, G, bf,
                                                       accumulate != 0 || !first[m], (hipStream_t)stream);
    if (err) return fail(RES_ERR_HIP, "grouped linear backward (weight): %s", err);
    first[m] = 0;
  }
  return RES_OK;
}

int resonator_grouped_linear_bwd_weight(const void* x, const void* dy, res_dtype_t dt, float* dW, int64_t N,
                                        int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* stream) {
  int rc = gl_check(N, d_in, d_out, G, dt);
  if (rc) return rc;
  if (!x || !dy || !dW) return fail(RES_ERR_INVALID_ARG, "x, dy and dW must be non-null");
  const size_t es = elt_size(dt);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(dW, 4))
    return fail(RES_ERR_MISALIGNED, "x and dy aligned to their element, dW to 4 bytes");
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * 4;
  if (overlap(dW, nw, x, nx) || overlap(dW, nw, dy, ny)) return fail(RES_ERR_INVALID_ARG, "dW must not overlap x or dy");
  const char* err = launch_grouped_linear_bwd_weight(x, dy, dW, N, d_in, d_out, G, dt == RES_BF16, accumulate != 0,
                                                     (hipStream_t)stream);
  if (err) return fail(RES_ERR_HIP, "grouped linear backward (weight): %s", err);
  return RES_OK;
}

int resonator_block_diag_weight(const void* W, res_dtype_t dt, int64_t d_in, int64_t d_out, int64_t G,
                                void* W_dense, void* stream) {
  if (d_in < 1 || d_out < 1 || G < 1 || d_in % G || d_out % G)
    return fail(RES_ERR_INVALID_ARG, "need d_in, d_out >= 1 and multiples of G >= 1");
  if (d_in * d_out > (1LL << 31)) return fail(RES_ERR_UNSUPPORTED, "d_in d_out must be <= 2^31");
  if (!dtype_ok(dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!W || !W_dense) return fail(RES_ERR_INVALID_ARG, "W and W_dense must be non-null");
  const size_t es = elt_size(dt);
  if (!aligned(W, es) || !aligned(W_dense, es)) return fail(RES_ERR_MISALIGNED, "W and W_dense must be aligned");
  if (overlap(W_dense, (size_t)(d_in * d_out) * es, W, (size_t)(d_in * (d_out / G)) * es))
    return fail(RES_ERR_INVALID_ARG, "W_dense must not overlap W");
  const hipError_t e = launch_block_diag(W, W_dense, d_in, d_out, G, dt == RES_BF16, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "block-diagonal weight launch");
}

size_t resonator_grouped_linear_bwd_weight_split_workspace_bytes(int64_t N, int64_t d_in, int64_t d_out) {
  if (N < 1 || d_in < 1 || d_out < 1 || N >= (1LL << 31) || d_in * d_out > (1LL << 31)) return 0;
  return (size_t)(splitk_parts(N) * d_in * d_out) * sizeof(float);
}

int resonator_grouped_linear_bwd_weight_split(const void* x, const void* dy, res_dtype_t dt, float* dW, int64_t N,
                                              int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* ws,
                                              size_t ws_bytes, void* stream) {
  int rc = gl_check(N, d_in, d_out, G, dt);
  if (rc) return rc;
  if (d_in * d_out > (1LL << 31)) return fail(RES_ERR_UNSUPPORTED, "d_in d_out must be <= 2^31");
  if (!x || !dy || !dW) return fail(RES_ERR_INVALID_ARG, "x, dy and dW must be non-null");
  const size_t es = dt == RES_BF16 ? 2 : 4;
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(dW, 4))
    return fail(RES_ERR_MISALIGNED, "x and dy aligned to their element, dW to 4 bytes");
  const size_t need = resonator_grouped_linear_bwd_weight_split_workspace_bytes(N, d_in, d_out);
  if (!ws || ws_bytes < need)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", need, ws_bytes);
  if (!aligned(ws, 256)) return fail(RES_ERR_MISALIGNED, "workspace must be 256-byte aligned");
  const size_t nx = (size_t)(N * d_in) * es, ny = (size_t)(N * d_out) * es, nw = (size_t)(d_in * (d_out / G)) * 4;
  if (overlap(dW, nw, x, nx) || overlap(dW, nw, dy, ny) || overlap(ws, need, x, nx) || overlap(ws, need, dy, ny) ||
      overlap(ws, need, dW, nw))
    return fail(RES_ERR_INVALID_ARG, "dW and the workspace must not overlap x, dy or each other");
  const char* err = launch_grouped_linear_bwd_weight_splitk(x, dy, dW, N, d_in, d_out, G, dt == RES_BF16,
                                                            accumulate != 0, (float*)ws, (hipStream_t)stream);
  if (err) return fail(RES_ERR_HIP, "grouped linear backward (weight, split): %s", err);
  return RES_OK;
}

int resonator_block_diag_extract(const float* W_dense, int64_t d_in, int64_t d_out, int64_t G, float* W,
                                 int accumulate, void* stream) {
  if (G < 1 || d_in < 1 || d_out < 1 || d_in % G || d_out % G)
    return fail(RES_ERR_INVALID_ARG, "need d_in, d_out >= 1 and multiples of G >= 1");
  if (d_in * d_out > (1LL << 31)) return fail(RES_ERR_UNSUPPORTED, "d_in d_out must be <= 2^31");
  if (!W || !W_dense) return fail(RES_ERR_INVALID_ARG, "W and W_dense must be non-null");
  if (!aligned(W, 4) || !aligned(W_dense, 4)) return fail(RES_ERR_MISALIGNED, "W and W_dense must be 4-byte aligned");
  if (overlap(W, (size_t)(d_in * (d_out / G)) * 4, W_dense, (size_t)(d_in * d_out) * 4))
    return fail(RES_ERR_INVALID_ARG, "W must not overlap W_dense");
  const hipError_t e = launch_block_extract(W_dense, W, d_in, d_out, G, accumulate != 0, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "block-diagonal extract launch");
}

// ---------------------------------------------------------------------------
// Quadratic causal reference (kernel-tail baseline, Sec. 5.3)
// ---------------------------------------------------------------------------
size_t resonator_quadratic_reference_workspace_bytes(int64_t L, int64_t D) {
  if (L < 1 || D < 1 || L * D > (1LL << 31)) return 0;
  return quad_workspace_bytes(L, D);
}

int resonator_quadratic_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                  const float* gamma, const float* omega, const float* amp, const float* phase,
                                  void* ws, size_t ws_bytes, void* stream) {
  int rc = check_sizes(B, L, D, M, false);
  if (rc) return rc;
  if (B > 65535 || L * D > (1LL << 31))
    return fail(RES_ERR_UNSUPPORTED, "quadratic reference needs B <= 65535 and L D <= 2^31");
  if (!x || !y) return fail(RES_ERR_INVALID_ARG, "x and y must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  const size_t need = quad_workspace_bytes(L, D);
  if (!ws || ws_bytes < need)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", need, ws_bytes);
  if (!aligned(x, 4) || !aligned(y, 4) || !aligned(ws, 4))
    return fail(RES_ERR_MISALIGNED, "x, y and the workspace must be 4-byte aligned");
  const size_t n = (size_t)(B * L * D) * 4;
  if (overlap(y, n, x, n) || overlap(y, n, ws, need) || overlap(x, n, ws, need))
    return fail(RES_ERR_INVALID_ARG, "x, y and the workspace must not overlap");
  const hipError_t e = launch_quad_reference(x, y, B, L, D, M, gamma, omega, amp, phase, (float*)ws,
                                             (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "quadratic reference launch");
}

// ---------------------------------------------------------------------------
// FFT convolution (the paper's own prefill evaluation, Sec. 3.2) as a baseline
// ---------------------------------------------------------------------------
static int fft_check(int64_t B, int64_t L, int64_t D) {
  if (B < 1 || L < 1 || D < 1) return fail(RES_ERR_INVALID_ARG, "B, L and D must be >= 1");
  if (B > 65535 || D > 65535 * 32 || L > (1LL << 26) || B * D * (int64_t)(fft_next_pow2(L) + 2) > (1LL << 40) ||
      D * (int64_t)((fft_next_pow2(L) + 2 + 8191) / 8192) > (1LL << 31) - 1)
    return fail(RES_ERR_UNSUPPORTED, "FFT reference needs B <= 65535, L <= 2^26 and a padded buffer under 2^40");
  return RES_OK;
}

size_t resonator_fft_reference_workspace_bytes(int64_t B, int64_t L, int64_t D) {
  if (fft_check(B, L, D)) return 0;
  size_t bytes = 0;
  if (const char* e = fft_workspace_bytes(B, L, D, &bytes)) {
    fail(RES_ERR_HIP, "FFT plan: %s", e);
    return 0;
  }
  return bytes;
}

int resonator_fft_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                            const float* gamma, const float* omega, const float* amp, const float* phase, void* ws,
                            size_t ws_bytes, void* stream) {
  int rc = check_sizes(B, L, D, M, false);
  if (rc) return rc;
  if ((rc = fft_check(B, L, D))) return rc;
  if (!x || !y) return fail(RES_ERR_INVALID_ARG, "x and y must be non-null");
  if ((rc = check_params(gamma, omega, amp, phase))) return rc;
  size_t need = 0;
  if (const char* e = fft_workspace_bytes(B, L, D, &need)) return fail(RES_ERR_HIP, "FFT plan: %s", e);
  if (!ws || ws_bytes < need)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", need, ws_bytes);
  if (!aligned(x, 4) || !aligned(y, 4) || !aligned(ws, 256))
    return fail(RES_ERR_MISALIGNED, "x and y must be 4-byte and the workspace 256-byte aligned");
  const size_t n = (size_t)(B * L * D) * 4;
  if (overlap(y, n, x, n) || overlap(y, n, ws, need) || overlap(x, n, ws, need))
    return fail(RES_ERR_INVALID_ARG, "x, y and the workspace must not overlap");
  if (const char* e = launch_fft_reference(x, y, B, L, D, M, gamma, omega, amp, phase, ws, (hipStream_t)stream))
    return fail(RES_ERR_HIP, "FFT reference: %s", e);
  return RES_OK;
}

// ---------------------------------------------------------------------------
// Constrained parameterization (Sec. 3.1, last paragraph)
// ---------------------------------------------------------------------------
static int prm_check_n(int64_t n) {
  if (n < 1 || n > (1LL << 31)) return fail(RES_ERR_INVALID_ARG, "n must be in [1, 2^31] (got %lld)", (long long)n);
  return RES_OK;
}

int resonator_params_map(const float* theta_gamma, const float* theta_omega, int64_t n, float alpha_min,
                         float* gamma, float* omega, void* stream) {
  int rc = prm_check_n(n);
  if (rc) return rc;
  if (!theta_gamma || !theta_omega || !gamma || !omega)
    return fail(RES_ERR_INVALID_ARG, "theta_gamma, theta_omega, gamma and omega must be non-null");
  if (!(alpha_min >= 0.f) || !std::isfinite(alpha_min))
    return fail(RES_ERR_INVALID_ARG, "alpha_min must be finite and >= 0");
  for (const void* q : {(const void*)theta_gamma, (const void*)theta_omega, (const void*)gamma, (const void*)omega})
    if (!aligned(q, 4)) return fail(RES_ERR_MISALIGNED, "arrays must be 4-byte aligned");
  const size_t b = (size_t)n * 4;
  if (overlap(gamma, b, omega, b)) return fail(RES_ERR_INVALID_ARG, "gamma and omega must not overlap");
  const hipError_t e = launch_params_map(theta_gamma, theta_omega, n, alpha_min, gamma, omega, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "parameter map launch");
}

int resonator_params_map_bwd(const float* theta_gamma, const float* theta_omega, const float* dgamma,
                             const float* domega, int64_t n, float* dtheta_gamma, float* dtheta_omega,
                             void* stream) {
  int rc = prm_check_n(n);
  if (rc) return rc;
  if (!theta_gamma || !theta_omega || !dgamma || !domega || !dtheta_gamma || !dtheta_omega)
    return fail(RES_ERR_INVALID_ARG, "all arrays must be non-null");
  for (const void* q : {(const void*)theta_gamma, (const void*)theta_omega, (const void*)dgamma,
                        (const void*)domega, (const void*)dtheta_gamma, (const void*)dtheta_omega})
    if (!aligned(q, 4)) return fail(RES_ERR_MISALIGNED, "arrays must be 4-byte aligned");
  const size_t b = (size_t)n * 4;
  if (overlap(dtheta_gamma, b, dtheta_omega, b))
    return fail(RES_ERR_INVALID_ARG, "dtheta_gamma and dtheta_omega must not overlap");
  const hipError_t e = launch_params_map_bwd(theta_gamma, theta_omega, dgamma, domega, n, dtheta_gamma,
                                             dtheta_omega, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "parameter map backward launch");
}

int resonator_params_init(int64_t D, int64_t M, double hl_min, double hl_max, double per_min, double per_max,
                          float alpha_min, float* theta_gamma, float* theta_omega, void* stream) {
  if (D < 1 || M < 1 || D * M > (1LL << 31))
    return fail(RES_ERR_INVALID_ARG, "need D, M >= 1 and D M <= 2^31 (got D=%lld M=%lld)", (long long)D,
                (long long)M);
  if (!theta_gamma || !theta_omega) return fail(RES_ERR_INVALID_ARG, "theta_gamma and theta_omega must be non-null");
  if (!aligned(theta_gamma, 4) || !aligned(theta_omega, 4))
    return fail(RES_ERR_MISALIGNED, "arrays must be 4-byte aligned");
  if (!(hl_min > 0.0) || !(hl_max >= hl_min) || !(per_min >= 2.0) || !(per_max >= per_min) ||
      !std::isfinite(hl_max) || !std::isfinite(per_max) || !(alpha_min >= 0.f))
    return fail(RES_ERR_INVALID_ARG, "need 0 < hl_min <= hl_max, 2 <= per_min <= per_max, alpha_min >= 0");
  if (!(std::log(2.0) / hl_max > (double)alpha_min))
    return fail(RES_ERR_INVALID_ARG, "the longest half-life must map above alpha_min (ln 2 / hl_max > alpha_min)");
  const size_t b = (size_t)(D * M) * 4;
  if (overlap(theta_gamma, b, theta_omega, b))
    return fail(RES_ERR_INVALID_ARG, "theta_gamma and theta_omega must not overlap");
  const hipError_t e = launch_params_init(D, M, hl_min, hl_max, per_min, per_max, (double)alpha_min, theta_gamma,
                                          theta_omega, (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "parameter init launch");
}

int resonator_diagnostics(const float* gamma, const float* omega, const float* amp, const float* phase, int64_t D,
                          int64_t M, int64_t T, float* half_life, float* energy, float* spectrum, void* stream) {
  if (D < 1 || M < 1) return fail(RES_ERR_INVALID_ARG, "D and M must be >= 1");
  if ((energy || spectrum) && T < 1) return fail(RES_ERR_INVALID_ARG, "T must be >= 1 for energy or spectrum");
  if (D * M > (1LL << 40) || (energy && D * M * T > (1LL << 40)) || (spectrum && (T / 2 + 1) * D > (1LL << 40)))
    return fail(RES_ERR_UNSUPPORTED, "diagnostics larger than 2^40 entries");
  if (!gamma) return fail(RES_ERR_INVALID_ARG, "gamma must be non-null");
  if (spectrum && (!omega || !amp || !phase))
    return fail(RES_ERR_INVALID_ARG, "omega, amp and phase must be non-null for the spectrum");
  const float* ins[4] = {gamma, omega, amp, phase};
  float* outs[3] = {half_life, energy, spectrum};
  const size_t np = (size_t)(D * M) * 4;
  const size_t no[3] = {np, (size_t)(D * M * (T > 0 ? T : 0)) * 4, (size_t)((T / 2 + 1) * D) * 4};
  for (int o = 0; o < 3; ++o) {
    if (!outs[o]) continue;
    if (!aligned(outs[o], 4)) return fail(RES_ERR_MISALIGNED, "outputs must be 4-byte aligned");
    for (int i = 0; i < 4; ++i)
      if (ins[i] && overlap(outs[o], no[o], ins[i], np)) return fail(RES_ERR_INVALID_ARG, "outputs must not overlap the parameters");
    for (int q = o + 1; q < 3; ++q)
      if (outs[q] && overlap(outs[o], no[o], outs[q], no[q])) return fail(RES_ERR_INVALID_ARG, "outputs must not overlap");
  }
  for (int i = 0; i < 4; ++i)
    if (ins[i] && !aligned(ins[i], 4)) return fail(RES_ERR_MISALIGNED, "parameters must be 4-byte aligned");
  const hipError_t e = launch_diagnostics(gamma, omega, amp, phase, D, M, T, half_life, energy, spectrum,
                                          (hipStream_t)stream);
  return e == hipSuccess ? RES_OK : hip_fail(e, "diagnostics launch");
}

// ---------------------------------------------------------------------------
// Mixer epilogue (Sec. 3.4)
// ---------------------------------------------------------------------------
static int epi_check(int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K) {
  if (B < 1 || L < 1 || H < 1 || dh < 1)
    return fail(RES_ERR_INVALID_ARG, "B, L, H, dh must be >= 1 (got %lld %lld %lld %lld)", (long long)B,
                (long long)L, (long long)H, (long long)dh);
  if (H > EPI_H_MAX || K < 0 || K > EPI_K_MAX || H * dh > (1 << 24) || B * L > (1LL << 40))
    return fail(RES_ERR_UNSUPPORTED, "epilogue needs H <= %d, 0 <= K <= %d, H dh <= 2^24 (got H=%lld dh=%lld K=%lld)",
                EPI_H_MAX, EPI_K_MAX, (long long)H, (long long)dh, (long long)K);
  return RES_OK;
}

// channels a thread may move as one vector: the widest of 16 bytes, 8 bytes, two
// elements, one element that divides the head size and to which every
// activation pointer is aligned
static int epi_vec(int64_t dh, size_t es, std::initializer_list<const void*> ps) {
  for (int vec : {(int)(16 / es), (int)(8 / es), 2}) {
    if (vec < 2 || dh % vec) continue;
    bool ok = true;
    for (const void* p : ps) ok = ok && (!p || aligned(p, (size_t)vec * es));
    if (ok) return vec;
  }
  return 1;
}

size_t resonator_epilogue_workspace_bytes(int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K) {
  if (B < 1 || L < 1 || H < 1 || H > EPI_H_MAX || dh < 1 || K < 0 || K > EPI_K_MAX) return 0;
  return epi_workspace_bytes(B, L, H, dh, K);
}

int resonator_epilogue_fwd(const void* y, const void* gate, const void* v, res_dtype_t act_dt, void* z,
                           int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K, const float* Ct,
                           float lambda_c, const float* w, const float* s, void* stream) {
  int rc = epi_check(B, L, H, dh, K);
  if (rc) return rc;
  if (!dtype_ok(act_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!y || !gate || !z || !Ct) return fail(RES_ERR_INVALID_ARG, "y, gate, z and Ct must be non-null");
  if (K > 0 && (!v || !w || !s)) return fail(RES_ERR_INVALID_ARG, "v, w and s must be non-null when K > 0");
  const size_t es = elt_size(act_dt), n = (size_t)(B * L * H * dh) * es;
  if (!aligned(y, es) || !aligned(gate, es) || !aligned(z, es) || (K > 0 && !aligned(v, es)) || !aligned(Ct, 4) ||
      (w && !aligned(w, 4)) || (s && !aligned(s, 4)))
    return fail(RES_ERR_MISALIGNED, "activations aligned to their element, parameters to 4 bytes");
  if (overlap(z, n, y, n) || overlap(z, n, gate, n) || (K > 0 && overlap(z, n, v, n)))
    return fail(RES_ERR_INVALID_ARG, "z must not overlap y, gate or v");
  const int vec = epi_vec(dh, es, {y, gate, z, K > 0 ? v : nullptr});
  hipStream_t st = (hipStream_t)stream;
  auto a16 = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (epi_z_lds((int)H, (int)dh, (int)K, act_dt == RES_BF16) > 0 && a16(y) && a16(gate) && a16(z) &&
      (K == 0 || a16(v))) {  // one token's channel offset of every head per lane; bitwise the same z
    const hipError_t e =
        act_dt == RES_BF16
            ? launch_epi_z_fwd<bf16_t>(y, gate, v, z, B, L, (int)H, (int)K, Ct, lambda_c, w, s, device_cus(), st)
            : launch_epi_z_fwd<float>(y, gate, v, z, B, L, (int)H, (int)K, Ct, lambda_c, w, s, device_cus(), st);
    return e == hipSuccess ? RES_OK : hip_fail(e, "epilogue launch");
  }
  const hipError_t e =
      act_dt == RES_BF16
          ? launch_epi_fwd<bf16_t>(y, gate, v, z, B, L, (int)H, (int)dh, (int)K, Ct, lambda_c, w, s, vec, st)
          : launch_epi_fwd<float>(y, gate, v, z, B, L, (int)H, (int)dh, (int)K, Ct, lambda_c, w, s, vec, st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "epilogue launch");
}

int resonator_epilogue_proj_fwd(const void* y, const void* gate, const void* v, res_dtype_t act_dt, const void* Wo,
                                void* out, void* z, int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K,
                                int64_t d_out, const float* Ct, float lambda_c, const float* w, const float* s,
                                void* stream) {
  int rc = epi_check(B, L, H, dh, K);
  if (rc) return rc;
  if (!dtype_ok(act_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (d_out < 1 || d_out % H)
    return fail(RES_ERR_INVALID_ARG, "d_out (%lld) must be a positive multiple of H (%lld)", (long long)d_out,
                (long long)H);
  if (!y || !gate || !Wo || !out || !Ct) return fail(RES_ERR_INVALID_ARG, "y, gate, Wo, out and Ct must be non-null");
  if (K > 0 && (!v || !w || !s)) return fail(RES_ERR_INVALID_ARG, "v, w and s must be non-null when K > 0");
  const bool bf = act_dt == RES_BF16;
  if (epi_proj_lds((int)H, (int)dh, (int)K, d_out, bf) == 0)
    return fail(RES_ERR_UNSUPPORTED,
                "the fused epilogue takes H <= 8, dh = %d, K <= 4 and d_out/H of 16 or 32 (got H %lld, dh %lld, "
                "K %lld, d_out %lld)",
                bf ? 32 : 16, (long long)H, (long long)dh, (long long)K, (long long)d_out);
  const size_t es = elt_size(act_dt), n = (size_t)(B * L * H * dh) * es, no = (size_t)(B * L * d_out) * es;
  auto a16 = [](const void* p) { return p == nullptr || ((uintptr_t)p & 15) == 0; };
  if (!a16(y) || !a16(gate) || !a16(Wo) || !a16(out) || (K > 0 && !a16(v)) || !aligned(Ct, 4) ||
      (w && !aligned(w, 4)) || (s && !aligned(s, 4)))
    return fail(RES_ERR_MISALIGNED, "activations, Wo and out aligned to 16 bytes, parameters to 4 bytes");
  const size_t nw = (size_t)(dh * d_out) * es;
  if (overlap(out, no, y, n) || overlap(out, no, gate, n) || (K > 0 && overlap(out, no, v, n)) ||
      overlap(out, no, Wo, nw))
    return fail(RES_ERR_INVALID_ARG, "out must not overlap y, gate, v or Wo");
  if (z) {
    if (!a16(z)) return fail(RES_ERR_MISALIGNED, "z must be 16-byte aligned");
    if (overlap(z, n, y, n) || overlap(z, n, gate, n) || (K > 0 && overlap(z, n, v, n)) || overlap(z, n, Wo, nw) ||
        overlap(z, n, out, no))
      return fail(RES_ERR_INVALID_ARG, "z must not overlap y, gate, v, Wo or out");
  }
  hipStream_t st = (hipStream_t)stream;
  const hipError_t e =
      bf ? launch_epi_proj_fwd<bf16_t>(y, gate, v, Wo, out, z, B, L, (int)H, (int)K, d_out, Ct, lambda_c, w, s,
                                       device_cus(), st)
         : launch_epi_proj_fwd<float>(y, gate, v, Wo, out, z, B, L, (int)H, (int)K, d_out, Ct, lambda_c, w, s,
                                      device_cus(), st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "fused epilogue launch");
}

int resonator_epilogue_bwd(const void* y, const void* gate, const void* v, const void* dz, res_dtype_t act_dt,
                           void* dy, void* dgate, void* dv, int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K,
                           const float* Ct, float lambda_c, const float* w, const float* s, float* dCt,
                           float* dlambda_c, float* dw, float* ds, void* ws, size_t ws_bytes, void* stream) {
  int rc = epi_check(B, L, H, dh, K);
  if (rc) return rc;
  if (!dtype_ok(act_dt)) return fail(RES_ERR_INVALID_ARG, "unknown dtype code");
  if (!y || !gate || !dz || !dy || !dgate || !Ct || !dCt || !dlambda_c)
    return fail(RES_ERR_INVALID_ARG, "y, gate, dz, dy, dgate, Ct, dCt and dlambda_c must be non-null");
  if (K > 0 && (!v || !w || !s || !dv || !dw || !ds))
    return fail(RES_ERR_INVALID_ARG, "v, w, s, dv, dw and ds must be non-null when K > 0");
  const size_t need = epi_workspace_bytes(B, L, H, dh, K);
  if (!ws || ws_bytes < need)
    return fail(RES_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", need, ws_bytes);
  const size_t es = elt_size(act_dt), n = (size_t)(B * L * H * dh) * es;
  if (!aligned(y, es) || !aligned(gate, es) || !aligned(dz, es) || !aligned(dy, es) || !aligned(dgate, es) ||
      (K > 0 && (!aligned(v, es) || !aligned(dv, es))) || !aligned(ws, 256))
    return fail(RES_ERR_MISALIGNED, "activations aligned to their element, workspace to 256 bytes");
  for (const void* o : {(const void*)dy, (const void*)dgate, (const void*)(K > 0 ? dv : nullptr)}) {
    if (!o) continue;
    if (overlap(o, n, y, n) || overlap(o, n, gate, n) || overlap(o, n, dz, n) || (K > 0 && overlap(o, n, v, n)))
      return fail(RES_ERR_INVALID_ARG, "dy, dgate and dv must not overlap the inputs");
  }
  if (overlap(dy, n, dgate, n) || (K > 0 && (overlap(dv, n, dy, n) || overlap(dv, n, dgate, n))))
    return fail(RES_ERR_INVALID_ARG, "dy, dgate and dv must not overlap each other");
  const int vec = epi_vec(dh, es, {y, gate, dz, dy, dgate, K > 0 ? dv : nullptr});
  hipStream_t st = (hipStream_t)stream;
  float* part = (float*)ws;
  const hipError_t e =
      act_dt == RES_BF16
          ? launch_epi_bwd<bf16_t>(y, gate, v, dz, dy, dgate, dv, B, L, (int)H, (int)dh, (int)K, Ct, lambda_c, w,
                                   s, dCt, dlambda_c, dw, ds, part, vec, st)
          : launch_epi_bwd<float>(y, gate, v, dz, dy, dgate, dv, B, L, (int)H, (int)dh, (int)K, Ct, lambda_c, w, s,
                                  dCt, dlambda_c, dw, ds, part, vec, st);
  return e == hipSuccess ? RES_OK : hip_fail(e, "epilogue backward launch");
}

}  // extern "C"

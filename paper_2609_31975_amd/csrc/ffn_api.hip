// Host side of the C ABI declared in include/ffn_sparse.h: argument checks,
// workspace carve-up and kernel sequencing.  No allocation, no synchronization on the
// forward path.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "ffn_internal.h"
#include "ffn_sparse.h"

namespace ffn {

thread_local GateTiming g_gate_timing;
std::atomic<uint64_t> g_z_wait{kZWaitTicks};
uint64_t z_wait_ticks() { return g_z_wait.load(std::memory_order_relaxed); }

namespace {
constexpr size_t kAlign = 256;
constexpr int64_t kMaxElems = (int64_t)1 << 31;  // kernels index rows with 32-bit chunk counts

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
}  // namespace

size_t workspace_layout(int T, int d, int d_ff, int r, void* base, Workspace* out) {
  Workspace w{};
  w.nseg = 0;
  w.slots = d_ff;
  w.tc = T < kTokChunk ? T : kTokChunk;
  w.r = r;
  size_t off = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) {
    char* p = b ? b + off : nullptr;
    off += round_up(bytes);
    return p;
  };
  w.meta = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 64));
  // right after meta, so that calls of any token count with one rank find their slots in the
  // same place
  w.zslot = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * (size_t)(r > 0 ? r : 1)));
  w.seg_count = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)d_ff));
  w.seg_idx = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)w.slots));
  w.seg_act = reinterpret_cast<float*>(take(sizeof(float) * (size_t)w.tc * w.slots));
  w.seg_zval = reinterpret_cast<float*>(take(sizeof(float) * (size_t)w.tc * w.slots));
  const size_t bt = w.tc >= 2 ? (size_t)w.tc : 0;  // matrix-core path only
  w.z = reinterpret_cast<float*>(take(sizeof(float) * (bt ? 2 : 1) * (size_t)w.tc * (r > 0 ? r : 1)));
  w.zsq = reinterpret_cast<float*>(take(sizeof(float) * (size_t)(r > 0 ? r : 1)));
  w.gx = reinterpret_cast<float*>(take(sizeof(float) * (r > 0 ? (size_t)w.tc * d_ff : 1)));
  w.zf = reinterpret_cast<uint4*>(take(sizeof(uint4) * 2 * ((bt + 15) / 16) * 2 * kWave * (size_t)batched_segments(d_ff)));
  const size_t xs_frags = bt >= (size_t)kPreSplitMin ? (size_t)((d + 31) / 32) * ((bt + 15) / 16) * kWave : 0;
  w.xs = reinterpret_cast<uint4*>(take(sizeof(uint4) * 2 * xs_frags));
  if (out) *out = w;
  return off;
}

namespace {

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_shape(int T, int d, int d_ff, int r, bool lopa) {
  if (T < 1 || d < 1 || d_ff < 1 || (lopa && r < 1)) return FFN_ERR_SHAPE;
  if ((int64_t)d_ff * d >= kMaxElems || (int64_t)T * d >= kMaxElems) return FFN_ERR_SHAPE;
  if (lopa && ((int64_t)r * d >= kMaxElems || (int64_t)d_ff * r >= kMaxElems)) return FFN_ERR_SHAPE;
  // the down kernel keeps one prefix entry per segment in LDS
  if (d_ff > (1 << 20)) return FFN_ERR_SHAPE;
  return FFN_OK;
}

struct Call {
  ffn_dtype_t wdt;
  int T, d, d_ff, r;  // r = 0: standard gating
  bool dense;
  const float* x;
  const void* gate;   // w_gate, or lopa_b for LoPA
  const void* lopa_a;
  const void* w_up;
  const void* w_down_t;
  float t;
  const ffn_options_t* opt;  // NULL: the default form
  float* y;
  void* ws;
  size_t ws_bytes;
  hipStream_t stream;
  bool quant_call = false;             // a *_q entry point (any ffn_dtype_t)
  const ffn_scales_t* scales = nullptr;
};

bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Checks ffn_options_t (see the header) and splits it into the gate kernels' Form and the
// norm's gain and eps (eps 0: no norm).
int check_options(const ffn_options_t* o, bool lopa, Form* form) {
  *form = Form{};
  form->z_wait = z_wait_ticks();
  if (!o) return FFN_OK;
  if ((o->act != FFN_ACT_RELU && o->act != FFN_ACT_RSPLUS) || (o->silu_up != 0 && o->silu_up != 1) ||
      (o->rms_norm != 0 && o->rms_norm != 1))
    return FFN_ERR_OPTION;
  if ((o->g_idx == nullptr) != (o->g_sign == nullptr)) return FFN_ERR_OPTION;
  if (!lopa && (o->g_idx || o->rms_norm || o->rms_gain)) return FFN_ERR_OPTION;
  if (o->rms_norm ? !(isfinite(o->rms_eps) && o->rms_eps > 0.f) : o->rms_gain != nullptr) return FFN_ERR_OPTION;
  if (!aligned4(o->g_idx) || !aligned4(o->rms_gain)) return FFN_ERR_ALIGN;
  form->act = o->act;
  form->silu_up = o->silu_up;
  form->g_idx = o->g_idx;
  form->g_sign = o->g_sign;
  if (o->rms_norm) {
    form->rms_gain = o->rms_gain;
    form->rms_eps = o->rms_eps;
  }
  return FFN_OK;
}

// The row scales of a quantized call, checked: FFN_OK with `out` filled, or an error.
int check_scales(const Call& c, bool lopa, Scales* out) {
  *out = Scales{};
  const bool quant = c.wdt == FFN_I8 || c.wdt == FFN_I4;
  if (!quant) return c.scales ? FFN_ERR_OPTION : FFN_OK;
  if (!c.scales) return FFN_ERR_NULL;
  const ffn_scales_t& s = *c.scales;
  if (!s.up || !s.down || (lopa ? (!s.lopa_a || !s.lopa_b) : !s.gate)) return FFN_ERR_NULL;
  if (!aligned4(s.up) || !aligned4(s.down) ||
      (lopa ? (!aligned4(s.lopa_a) || !aligned4(s.lopa_b)) : !aligned4(s.gate)))
    return FFN_ERR_ALIGN;
  *out = lopa ? Scales{nullptr, s.lopa_a, s.lopa_b, s.up, s.down} : Scales{s.gate, nullptr, nullptr, s.up, s.down};
  return FFN_OK;
}

// The host-side checks of a call's pointers, dtype and shape (not of the workspace when
// `with_ws` is false: the no-allocation entry point supplies its own).
int check_call(const Call& c, bool with_ws) {
  const bool lopa = c.r > 0;
  if (!c.x || !c.gate || !c.w_up || !c.w_down_t || !c.y || (with_ws && !c.ws) || (lopa && !c.lopa_a))
    return FFN_ERR_NULL;
  const bool quant = c.wdt == FFN_I8 || c.wdt == FFN_I4;
  if ((c.wdt != FFN_F32 && c.wdt != FFN_BF16 && !quant) || (quant && !c.quant_call)) return FFN_ERR_DTYPE;
  const int sc = check_shape(c.T, c.d, c.d_ff, c.r, lopa);
  if (sc != FFN_OK) return sc;
  if (c.wdt == FFN_I4 && (c.d % 2 != 0 || (lopa && c.r % 2 != 0))) return FFN_ERR_SHAPE;
  if (!aligned(c.x) || !aligned(c.gate) || !aligned(c.w_up) || !aligned(c.w_down_t) || !aligned(c.y) ||
      (with_ws && !aligned(c.ws)) || (lopa && !aligned(c.lopa_a)))
    return FFN_ERR_ALIGN;
  return FFN_OK;
}

int run(const Call& c) {
  const bool lopa = c.r > 0;
  const int cc = check_call(c, true);
  if (cc != FFN_OK) return cc;
  Form form;
  const int so = check_options(c.opt, lopa, &form);
  if (so != FFN_OK) return so;
  Scales scales;
  const int ss = check_scales(c, lopa, &scales);
  if (ss != FFN_OK) return ss;
  Workspace ws;
  if (c.ws_bytes < workspace_layout(c.T, c.d, c.d_ff, c.r, c.ws, &ws)) return FFN_ERR_WORKSPACE;

  // tokens run in passes of up to kTokChunk; each pass is an independent FFN call
  for (int t0 = 0; t0 < c.T; t0 += kTokChunk) {
    Shape sh{c.T - t0 < kTokChunk ? c.T - t0 : kTokChunk, c.d, c.d_ff, c.r, (int)c.wdt, scales};
    const float* x = c.x + (size_t)t0 * c.d;
    float* y = c.y + (size_t)t0 * c.d;
    const Gate g = lopa ? Gate::LoPA : Gate::Standard;
    hipError_t e = hipSuccess;
    if (batched_ok(sh, g)) {
      e = launch_batched(sh, g, c.dense, form, x, c.lopa_a, c.gate, c.w_up, c.w_down_t, c.t, ws, y, c.stream);
    } else {
      // z = A x: in the gate kernel where it can (its down kernel then clears the z slots)
      const bool fz = lopa && lopa_fuses_z(sh, form);
      if (lopa && !fz) e = launch_lopa_z(sh, form, x, c.lopa_a, ws, c.stream);
      if (e == hipSuccess)
        e = launch_gate_up(sh, g, c.dense, form, x, c.gate, c.w_up, c.t, ws, y, c.stream, fz ? c.lopa_a : nullptr);
      if (e == hipSuccess) e = launch_down(sh, c.dense, c.w_down_t, ws, y, c.stream, fz);
    }
    if (e != hipSuccess) return FFN_ERR_HIP;
  }
  return FFN_OK;
}

// ------------------------------------------------------------------ the no-allocation entry point
// Its workspace: a file-scope device array, one copy per GPU the library runs on, held until
// the process ends.  In host code `scratch` names a host-side stand-in, so its device
// address is taken once per device with hipGetSymbolAddress and kept in g_scratch.
constexpr size_t kScratchBytes = size_t(16) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The scratch array's device address on the current device (set up on the first call made
// with that device current), or null if the runtime cannot give it.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace
}  // namespace ffn

using ffn::Call;

extern "C" {

size_t ffn_workspace_bytes(int T, int d, int d_ff, int r) {
  if (ffn::check_shape(T, d, d_ff, r, r > 0) != FFN_OK || r < 0) return 0;
  return ffn::workspace_layout(T, d, d_ff, r, nullptr, nullptr);
}

int ffn_dense_forward(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                      const void* w_up, const void* w_down_t, float t, float* y, void* ws, size_t ws_bytes,
                      hipStream_t stream) {
  return ffn::run(
      Call{wdt, T, d, d_ff, 0, true, x, w_gate, nullptr, w_up, w_down_t, t, nullptr, y, ws, ws_bytes, stream});
}

int ffn_sparse_forward(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                       const void* w_up, const void* w_down_t, float t, float* y, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  return ffn::run(
      Call{wdt, T, d, d_ff, 0, false, x, w_gate, nullptr, w_up, w_down_t, t, nullptr, y, ws, ws_bytes, stream});
}

int ffn_lopa_sparse_forward(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x, const void* lopa_a,
                            const void* lopa_b, const void* w_up, const void* w_down_t, float t, float* y, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(
      Call{wdt, T, d, d_ff, r, false, x, lopa_b, lopa_a, w_up, w_down_t, t, nullptr, y, ws, ws_bytes, stream});
}

int ffn_lopa_dense_forward(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x, const void* lopa_a,
                           const void* lopa_b, const void* w_up, const void* w_down_t, float t, float* y, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(
      Call{wdt, T, d, d_ff, r, true, x, lopa_b, lopa_a, w_up, w_down_t, t, nullptr, y, ws, ws_bytes, stream});
}

int ffn_sparse_forward_noalloc(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                               const void* w_up, const void* w_down_t, float t, float* y, hipStream_t stream) {
  Call c{wdt, T, d, d_ff, 0, false, x, w_gate, nullptr, w_up, w_down_t, t, nullptr, y, nullptr, 0, stream};
  const int cc = ffn::check_call(c, false);
  if (cc != FFN_OK) return cc;
  if (ffn::workspace_layout(T, d, d_ff, 0, nullptr, nullptr) > ffn::kScratchBytes) return FFN_ERR_WORKSPACE;
  c.ws = ffn::scratch_on_current_device();
  if (!c.ws) return FFN_ERR_HIP;
  c.ws_bytes = ffn::kScratchBytes;
  return ffn::run(c);
}

int ffn_dense_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                         const void* w_up, const void* w_down_t, float t, const ffn_options_t* opt, float* y,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  return ffn::run(Call{wdt, T, d, d_ff, 0, true, x, w_gate, nullptr, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream});
}

int ffn_sparse_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                          const void* w_up, const void* w_down_t, float t, const ffn_options_t* opt, float* y,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  return ffn::run(
      Call{wdt, T, d, d_ff, 0, false, x, w_gate, nullptr, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream});
}

int ffn_lopa_sparse_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                               const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                               float t, const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(Call{wdt, T, d, d_ff, r, false, x, lopa_b, lopa_a, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream});
}

int ffn_lopa_dense_forward_ex(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                              const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                              float t, const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(Call{wdt, T, d, d_ff, r, true, x, lopa_b, lopa_a, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream});
}

int ffn_dense_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                        const void* w_up, const void* w_down_t, const ffn_scales_t* scales, float t,
                        const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes, hipStream_t stream) {
  return ffn::run(Call{wdt, T, d, d_ff, 0, true, x, w_gate, nullptr, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream,
                       true, scales});
}

int ffn_sparse_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, const float* x, const void* w_gate,
                         const void* w_up, const void* w_down_t, const ffn_scales_t* scales, float t,
                         const ffn_options_t* opt, float* y, void* ws, size_t ws_bytes, hipStream_t stream) {
  return ffn::run(Call{wdt, T, d, d_ff, 0, false, x, w_gate, nullptr, w_up, w_down_t, t, opt, y, ws, ws_bytes,
                       stream, true, scales});
}

int ffn_lopa_sparse_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                              const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                              const ffn_scales_t* scales, float t, const ffn_options_t* opt, float* y, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(Call{wdt, T, d, d_ff, r, false, x, lopa_b, lopa_a, w_up, w_down_t, t, opt, y, ws, ws_bytes,
                       stream, true, scales});
}

int ffn_lopa_dense_forward_q(ffn_dtype_t wdt, int T, int d, int d_ff, int r, const float* x,
                             const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                             const ffn_scales_t* scales, float t, const ffn_options_t* opt, float* y, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  if (r < 1) return FFN_ERR_SHAPE;
  return ffn::run(Call{wdt, T, d, d_ff, r, true, x, lopa_b, lopa_a, w_up, w_down_t, t, opt, y, ws, ws_bytes, stream,
                       true, scales});
}

int ffn_active_set(const void* ws, int T, int d, int d_ff, int r, int32_t* n_union, int32_t* idx_host,
                   float* act_host, hipStream_t stream) {
  if (!ws || !n_union || !idx_host) return FFN_ERR_NULL;
  if (r < 0 || ffn::check_shape(T, d, d_ff, r, r > 0) != FFN_OK || T > ffn::kTokChunk) return FFN_ERR_SHAPE;
  ffn::Workspace w;
  ffn::workspace_layout(T, d, d_ff, r, const_cast<void*>(ws), &w);
  if (hipStreamSynchronize(stream) != hipSuccess) return FFN_ERR_HIP;
  int32_t nseg = 0;
  if (hipMemcpy(&nseg, w.meta, sizeof nseg, hipMemcpyDeviceToHost) != hipSuccess) return FFN_ERR_HIP;
  if (nseg < 1 || nseg > d_ff) return FFN_ERR_HIP;  // workspace does not hold a finished call
  std::vector<int32_t> cnt(nseg), idx(w.slots);
  std::vector<float> act;
  if (hipMemcpy(cnt.data(), w.seg_count, sizeof(int32_t) * nseg, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(idx.data(), w.seg_idx, sizeof(int32_t) * w.slots, hipMemcpyDeviceToHost) != hipSuccess)
    return FFN_ERR_HIP;
  if (act_host) {
    act.resize((size_t)T * w.slots);
    if (hipMemcpy(act.data(), w.seg_act, sizeof(float) * act.size(), hipMemcpyDeviceToHost) != hipSuccess)
      return FFN_ERR_HIP;
  }
  int n = 0;
  const ffn::Split segs(d_ff, nseg);
  for (int s = 0; s < nseg; ++s) {
    const int row0 = segs.start(s), row1 = segs.start(s + 1);
    if (cnt[s] < 0 || cnt[s] > row1 - row0) return FFN_ERR_HIP;  // workspace does not hold a finished call
    for (int e = 0; e < cnt[s]; ++e) {
      const int slot = row0 + e;
      if (act_host)
        for (int tau = 0; tau < T; ++tau) act_host[(size_t)tau * d_ff + n] = act[(size_t)tau * w.slots + slot];
      idx_host[n++] = idx[slot];
    }
  }
  *n_union = n;
  return FFN_OK;
}

int ffn_workspace_active(const void* ws, int T, int d, int d_ff, int r, const int32_t** meta,
                         const int32_t** seg_count, const int32_t** idx, const float** act) {
  if (!ws || !meta || !seg_count || !idx || !act) return FFN_ERR_NULL;
  if (r < 0 || ffn::check_shape(T, d, d_ff, r, r > 0) != FFN_OK || T > ffn::kTokChunk) return FFN_ERR_SHAPE;
  ffn::Workspace w;
  ffn::workspace_layout(T, d, d_ff, r, const_cast<void*>(ws), &w);
  *meta = w.meta;
  *seg_count = w.seg_count;
  *idx = w.seg_idx;
  *act = w.seg_act;
  return FFN_OK;
}

int ffn_time_next_gate_kernel(hipEvent_t start, hipEvent_t stop) {
  if ((start == nullptr) != (stop == nullptr)) return FFN_ERR_NULL;
  ffn::g_gate_timing = ffn::GateTiming{start, stop};
  return FFN_OK;
}

int ffn_set_z_wait_ticks(uint64_t ticks) {
  ffn::g_z_wait.store(ticks, std::memory_order_relaxed);
  return FFN_OK;
}

const char* ffn_status_string(int status) {
  switch (status) {
    case FFN_OK: return "ok";
    case FFN_ERR_NULL: return "null pointer argument";
    case FFN_ERR_SHAPE: return "invalid shape";
    case FFN_ERR_DTYPE: return "invalid weight dtype";
    case FFN_ERR_ALIGN: return "pointer not aligned (16 bytes; g_idx and rms_gain 4 bytes)";
    case FFN_ERR_WORKSPACE: return "workspace too small";
    case FFN_ERR_HIP: return "HIP launch or copy failed";
    case FFN_ERR_OPTION: return "invalid ffn_options_t field";
    default: return "unknown status";
  }
}

}  // extern "C"

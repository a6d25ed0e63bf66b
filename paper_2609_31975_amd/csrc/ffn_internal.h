// Internal declarations shared by the kernels and the host dispatcher of the
// sparse-FFN library (gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ffn {

constexpr int kWave = 64;
constexpr int kSegMax = 64;       // most gate rows per segment (one 64-lane ballot)
constexpr int kSegGeneric = 32;   // rows per segment of the element-wise kernels
constexpr int kBlock = 256;       // threads per workgroup for every kernel
constexpr int kTokChunk = 64;     // tokens per pass; a larger batch runs as several passes
constexpr int kListWindow = 1024; // active entries staged in LDS at a time by the down kernel
constexpr int kPreSplitMin = 17;  // batches of more than one 16-token tile get their tokens pre-split
// Tag of a published z value (a signalling-NaN bit pattern, which no arithmetic produces and
// none of the workspace's other data holds), and the most z components the single-token gate
// kernel computes itself (8 a thread).
constexpr uint32_t kZTag = 0x7FA5A5A5u;
constexpr int kFusedZMax = 8 * 256;
// How long a gate workgroup waits for the z components of the others before it computes the
// missing ones itself: 100 us of the 100 MHz constant clock (wall_clock64).
constexpr uint64_t kZWaitTicks = 10000;

// Balanced split of n items into `parts` ranges; range w is [start(w), start(w + 1)).
// The first n % parts ranges hold n / parts + 1 items, the others n / parts.  32-bit
// arithmetic only (0 <= n < 2^31, parts >= 1): the one division happens when the split
// is built, so a kernel pays it once and every range bound is a multiply and a min.
struct Split {
  uint32_t q, rem;
  __host__ __device__ Split(int n, int parts)
      : q((uint32_t)n / (uint32_t)parts), rem((uint32_t)n - (uint32_t)n / (uint32_t)parts * (uint32_t)parts) {}
  __host__ __device__ int start(int w) const {
    const uint32_t u = (uint32_t)w;
    return (int)(u * q + (u < rem ? u : rem));
  }
  // the range that holds item i, 0 <= i < n
  __host__ __device__ int of(int i) const {
    const uint32_t u = (uint32_t)i, big = rem * (q + 1);
    return (int)(u < big ? u / (q + 1) : rem + (u - big) / q);
  }
};

// Workspace carve-up for one pass of up to `tc` tokens.  Every region starts on a
// 256-byte boundary.  The neurons are split into nseg row-balanced segments (chosen
// per call by the gate launcher and recorded in meta[0]): segment w covers rows
// [Split(d_ff, nseg).start(w), ....start(w + 1)), and its active neurons occupy the
// slots from its first row on: slot start(w) + e holds its e-th active neuron
// (ascending), for e < seg_count[w].  slots = d_ff.
struct Workspace {
  int nseg;
  int slots;
  int tc;
  int r;
  int32_t* meta;       // [64]             meta[0] = nseg of the last call
  uint64_t* zslot;     // [r]              LoPA z of one token as published by the gate kernel that
                       //                  computes it (kZTag in the high word, the fp32 value in
                       //                  the low one); all-zero tags between calls (LoPA only)
  int32_t* seg_count;  // [d_ff]           (at most d_ff segments)
  int32_t* seg_idx;    // [slots]          neuron index
  float* seg_act;      // [tc][slots]      h - t for the token, 0 where inactive
  float* seg_zval;     // [tc][slots]      act * <w_up[i], x_tau>
  float* z;            // [tc][r]          LoPA intermediate A x (LoPA only); for tc >= 2
                       //                  two partial copies [2][tc][r]
  float* zsq;          // [r]              squares of z (single-token LoPA path with RMSNorm)
  float* gx;           // [tc][d_ff]       G x per token (LoPA with G, single-token and
                       //                  matrix-core paths; written by the z kernel)
  uint4* zf;           // [2 batched_segments(d_ff)][ceil(tc / 16)][2][64]  zval fragments of the
                       //                  down product, hi and lo planes of 64 lanes per fragment
                       //                  group and token tile (matrix-core path, tc >= 2)
  uint4* xs;           // [2][ceil(d / 32)][ceil(tc / 16)][64]  tokens split into bf16 hi / lo
                       //                  matrix-core fragments (tc >= kPreSplitMin, else empty)
};

size_t workspace_layout(int T, int d, int d_ff, int r, void* base, Workspace* out);

// Kernel launch parameters decided on the host.
// Row scales of quantized weights (FFN_I8 / FFN_I4): one fp32 per stored matrix row; all
// null for fp32 / bf16 weights.
struct Scales {
  const float* gate = nullptr;  // [d_ff]
  const float* a = nullptr;     // [r]
  const float* b = nullptr;     // [d_ff]
  const float* up = nullptr;    // [d_ff]
  const float* down = nullptr;  // [d_ff]
};

struct Shape {
  int T, d, d_ff, r;
  int wdt;    // 0 fp32, 1 bf16, 2 int8, 3 int4 (the ffn_dtype_t values)
  Scales sc;  // row scales (int8 / int4)
};

enum class Gate { Standard, LoPA };

// Compile-time form of a gate kernel: the default form, the full form's activations
// only, or (LoPA) also G and RMSNorm.
enum FormKind : int { kFormDefault = 0, kFormAct = 1, kFormLoPA = 2 };

// The paper's full FFN form (from ffn_options_t, checked on the host): the activation,
// SiLU on the W_up output, LoPA's fixed term G and RMSNorm of z.
struct Form {
  int act = 0;                     // 0 shifted ReLU, 1 shifted R-S+
  int silu_up = 0;                 // 1: SiLU on the W_up output
  const int32_t* g_idx = nullptr;  // G's column per row (null: G = 0, and g_sign null)
  const int8_t* g_sign = nullptr;  // G's value per row
  const float* rms_gain = nullptr;  // RMSNorm gains over z (null: ones)
  float rms_eps = 0.f;              // > 0: RMSNorm between the LoPA factors
  uint64_t z_wait = kZWaitTicks;    // single-token LoPA: the gate workgroups' bounded wait for z
  bool full() const { return act != 0 || silu_up != 0 || g_idx != nullptr || rms_eps > 0.f; }
  int kind() const { return g_idx != nullptr || rms_eps > 0.f ? kFormLoPA : full() ? kFormAct : kFormDefault; }
};

// Events for the next gate-kernel launch on this host thread (benchmark hook).
struct GateTiming {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
extern thread_local GateTiming g_gate_timing;

// The bounded wait for z of the calls that follow (ffn_set_z_wait_ticks; kZWaitTicks unless set).
uint64_t z_wait_ticks();

// Launchers (return hipSuccess or the launch error).  Every launcher enqueues on `s`.
// With form.rms_eps > 0 on the single-token path, z is stored times the RMSNorm gains and
// its squares go to ws.zsq; the gate kernel then scales each gate value by the norm.
hipError_t launch_lopa_z(const Shape& sh, const Form& form, const float* x, const void* lopa_a, const Workspace& ws,
                         hipStream_t s);
// RMSNorm on z in place (Section 3.3): the `parts` partial copies [parts][tc][r] of each
// token's z are summed into copy 0, scaled by gain / sqrt(mean z^2 + eps), and the other
// copies are zeroed, so the gate kernels read the normalized z unchanged.
hipError_t launch_rms_norm(float* z, int parts, int tc, int T, int r, const float* gain, float eps,
                           hipStream_t s);
// Also clears y[0 .. T*d) and sets ws.nseg / meta[0] for the down kernel.  With
// form.rms_eps > 0 (LoPA) z is normalised first: inside the single-token gate kernel,
// else by launch_rms_norm.
// lopa_a (only where lopa_fuses_z holds): the gate kernel computes z = A x itself.
hipError_t launch_gate_up(const Shape& sh, Gate g, bool dense, const Form& form, const float* x,
                          const void* gate_w, const void* w_up, float t, Workspace& ws, float* y, hipStream_t s,
                          const void* lopa_a = nullptr);
hipError_t launch_down(const Shape& sh, bool dense, const void* w_down_t, const Workspace& ws, float* y,
                       hipStream_t s, bool clear_zslots = false);
// The single-token LoPA gate kernel computes z = A x itself (no z kernel before it; the down
// kernel then clears ws.zslot): fp32 / bf16 rows of the single-token kernels, r <= kFusedZMax.
bool lopa_fuses_z(const Shape& sh, const Form& form);

// Matrix-core path for batches of 2..64 tokens with bf16 weights (ffn_batched.hip):
// the whole call (LoPA z, gate + union + W_up, down), clearing y first.
bool batched_ok(const Shape& sh, Gate g);
int batched_segments(int d_ff);
// form.rms_eps > 0: RMSNorm on z between the LoPA factors.
hipError_t launch_batched(const Shape& sh, Gate g, bool dense, const Form& form, const float* x,
                          const void* lopa_a, const void* gate_w, const void* w_up, const void* w_down_t, float t,
                          Workspace& ws, float* y, hipStream_t s);

}  // namespace ffn

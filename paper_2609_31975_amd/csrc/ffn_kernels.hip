// gfx950 kernels of the activation-sparse FFN forward pass.
//
// Data flow of one pass (paper Section 3.1: the gate is computed in full, zeros of
// A(W1 x) are known before W3 and W2 are touched; Section 3.3: LoPA gate B (A x)):
//
//   [LoPA only] k_lopa_z*     z = A x                               -> ws.z
//   k_gate_up*                one workgroup per row-balanced segment of neurons:
//                             h = W_gate x (or B z), 64-lane ballot compaction of the
//                             neurons with h > t (union over tokens), then the W_up
//                             row dot products of exactly those neurons:
//                             act = h - t, zval = act * <w_up[i], x>
//                             -> seg_count / seg_idx / seg_act / seg_zval; clears y
//   k_down*                   y += zval_k * w_down_t[idx_k] over the listed neurons;
//                             one workgroup per (row chunk, 1 KB column slice), fp32
//                             atomics into y across row chunks.
//
// The compaction needs no atomics and no inter-workgroup waits: each segment writes
// its own count and an ascending list, and readers find a segment's list from its
// first row.
#include <hip/hip_ext.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace ffn {
namespace {

// ------------------------------------------------------------------ row-dot helpers
// A row of C 16-byte chunks is covered by a group of `lpr` lanes; lane q of the group
// owns chunks q, q + lpr, ..., q + (CPL-1) lpr.  A wave covers 64/lpr rows at once.
template <class W, int CPL>
__device__ __forceinline__ void load_vec(const float* __restrict__ v, int C, int q, int lpr,
                                         float (&r)[CPL][W::EPC]) {
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = q + c * lpr;
    if (ch < C) {
      const float4* p = reinterpret_cast<const float4*>(v + (size_t)ch * W::EPC);
#pragma unroll
      for (int e4 = 0; e4 < W::EPC / 4; ++e4) {
        const float4 f = p[e4];
        r[c][4 * e4 + 0] = f.x;
        r[c][4 * e4 + 1] = f.y;
        r[c][4 * e4 + 2] = f.z;
        r[c][4 * e4 + 3] = f.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < W::EPC; ++e) r[c][e] = 0.f;
    }
  }
}

template <class W, int CPL>
__device__ __forceinline__ float lane_dot(const uint4 (&b)[CPL], const float (&v)[CPL][W::EPC]) {
  float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    float f[W::EPC];
    unpack(W{}, b[c], f);
#pragma unroll
    for (int e = 0; e < W::EPC; e += 2) {
      acc0 = fmaf(f[e], v[c][e], acc0);
      acc1 = fmaf(f[e + 1], v[c][e + 1], acc1);
    }
  }
  return acc0 + acc1;
}

// Dot products <rows, v> for rows picked by `row_of(k)`, k in [0, n), of a matrix of
// `bytes` bytes (< 2^31): each wave takes passes of 64/lpr rows (passes wave, wave + 4,
// ...).  For rows of at most 8 chunks per lane and more than one pass per wave, two
// register sets alternate, the loads of the next pass issued before the current pass is
// reduced; the loads are raw buffer loads (out-of-range offsets past the last pass), so
// every pass issues the same loads and the load-counter waits are exact.  A pair of
// passes always runs both halves (a pass past the last one loads nothing and sinks
// nothing) and the exit test closes the pair, so no load sits on a conditional path.
// `sink(k, value)` runs on lane q == 0.
template <class W, int CPL>
__device__ __forceinline__ void load_pass(const Buf& mb, int C, int q, int lpr, bool ok, int row, uint4 (&b)[CPL]) {
  const uint32_t base = ok ? 16u * (uint32_t)row * (uint32_t)C : kOOB;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = q + c * lpr;
    b[c] = ldb_nt(mb, (ok && ch < C) ? base + 16u * (uint32_t)ch : kOOB);
  }
}

template <class W, int CPL, class RowOf, class Sink>
__device__ __forceinline__ void dot_rows(const uint4* __restrict__ mat, uint32_t bytes, int C, int lpr, int lpr_log2,
                                         int n, const float (&v)[CPL][W::EPC], RowOf row_of, Sink sink) {
  constexpr int kWaves = kBlock / kWave;
  const Buf mb = make_buf(mat, bytes);
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const int q = lane & (lpr - 1), p = lane >> lpr_log2;
  const int rpp = kWave >> lpr_log2;
  const int npass = (n + rpp - 1) / rpp;
  if (wave >= npass) return;
  auto load = [&](uint4 (&b)[CPL], int pass) {
    const int k = pass * rpp + p;
    const bool ok = pass < npass && k < n;
    load_pass<W, CPL>(mb, C, q, lpr, ok, ok ? row_of(k) : 0, b);
  };
  auto finish = [&](const uint4 (&b)[CPL], int pass) {
    const int k = pass * rpp + p;
    const float sum = group_sum(lane_dot<W, CPL>(b, v), lpr);
    if (q == 0 && k < n) sink(k, sum);
  };
  uint4 b0[CPL];
  load(b0, wave);
  if (wave + kWaves >= npass) {  // a single pass: nothing to overlap
    finish(b0, wave);
    return;
  }
  if constexpr (CPL <= 8) {
    uint4 b1[CPL];
    for (int pass = wave;; pass += 2 * kWaves) {
      load(b1, pass + kWaves);
      issue_barrier();
      finish(b0, pass);
      load(b0, pass + 2 * kWaves);
      issue_barrier();
      finish(b1, pass + kWaves);
      if (pass + 2 * kWaves >= npass) break;
    }
  } else {
    for (int pass = wave;;) {
      finish(b0, pass);
      pass += kWaves;
      if (pass >= npass) break;
      load(b0, pass);
    }
  }
}

// Ballot compaction of one segment (run by the first wave): neurons whose gate value
// exceeds t (all neurons if `all`) get ascending ranks; their activation value (h - t,
// or its R-S+ with act = 1) is kept in LDS for the W_up phase and published with the
// neuron index.
__device__ __forceinline__ void compact_segment(const float* s_h, int nrows, int row0, int seg, float t, bool all,
                                                int act, int* s_list, float* s_act, int* s_cnt, int32_t* seg_count,
                                                int32_t* seg_idx, float* seg_act) {
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const bool valid = lane < nrows;
    const float h = valid ? s_h[lane] : 0.f;
    const bool on = h > t;  // NaN compares false: inactive
    const bool sel = valid && (all || on);
    const uint64_t m = __ballot(sel);
    const int rank = rank_in_mask(m);
    if (sel) {
      const float a = on ? gate_value(act, h - t) : 0.f;
      s_list[rank] = lane;
      s_act[rank] = a;
      seg_idx[row0 + rank] = row0 + lane;
      seg_act[row0 + rank] = a;
    }
    if (lane == 0) {
      const int cnt = __popcll(m);
      *s_cnt = cnt;
      seg_count[seg] = cnt;
    }
  }
}

// components of z (or of its squares) a thread keeps in registers for RMSNorm
constexpr int kNormRegs = 4;

// ------------------------------------------------------------------ fast kernels, T = 1
// z = A x for one token (rows of A: C chunks); one pass of 64/lpr rows per wave.
// NORM (RMSNorm between the factors, Section 3.3): z_k is stored times gain_k and z_k^2
// goes to zsq, from which the gate kernel takes the norm; the norm being one scalar per
// token, it scales each gate value B (gain . z) after the dot product.
template <class W, int CPL, bool NORM>
__global__ __launch_bounds__(kBlock) void k_lopa_z_t1(const float* __restrict__ x, const uint4* __restrict__ A,
                                                      int C, int lpr, int lpr_log2, int r, float* __restrict__ z,
                                                      const float* __restrict__ gain, float* __restrict__ zsq,
                                                      GWork gw) {
  if (g_precompute(gw)) return;
  float xr[CPL][W::EPC];
  load_vec<W, CPL>(x, C, lane_id() & (lpr - 1), lpr, xr);
  const int rows_per_block = (kBlock / kWave) * (kWave >> lpr_log2);
  const int k0 = blockIdx.x * rows_per_block;
  const int n = min(rows_per_block, r - k0);
  dot_rows<W, CPL>(A, 16u * (uint32_t)r * (uint32_t)C, C, lpr, lpr_log2, n, xr, [&](int k) { return k0 + k; },
                   [&](int k, float s) {
                     if constexpr (NORM) {
                       z[k0 + k] = gain ? s * gain[k0 + k] : s;
                       zsq[k0 + k] = s * s;
                     } else {
                       z[k0 + k] = s;
                     }
                   });
}

// One segment: gate values, compaction, W_up dots of the selected neurons.
// LOPA: the gate rows are B [d_ff][r] against z; otherwise W_gate [d_ff][d] against x.
// DENSE: every neuron of the segment is selected (act = max(h - t, 0)).
// FORM (a FormKind): the paper's full form (`form`): the activation value, SiLU on the
// W_up output and, with kFormLoPA, the fixed term G and RMSNorm of z.
template <class W, bool LOPA, bool DENSE, int CPLG, int CPLU, int FORM>
__global__ __launch_bounds__(kBlock) void k_gate_up_t1(const float* __restrict__ x, const float* __restrict__ z,
                                                       const uint4* __restrict__ gate_w, int Cg, int lprg,
                                                       int lprg_log2, const uint4* __restrict__ w_up, int Cu,
                                                       int lpru, int lpru_log2, int d_ff, int nseg, float t,
                                                       int32_t* __restrict__ meta, int32_t* __restrict__ seg_count,
                                                       int32_t* __restrict__ seg_idx, float* __restrict__ seg_act,
                                                       float* __restrict__ seg_zval, float* __restrict__ y, int d,
                                                       Form form, const float* __restrict__ zsq,
                                                       const float* __restrict__ gx) {
  constexpr bool FULL = FORM != kFormDefault, EXTRA = LOPA && FORM == kFormLoPA;
  __shared__ float s_h[kSegMax];
  __shared__ float s_ss[kBlock / kWave];
  __shared__ int s_list[kSegMax];
  __shared__ float s_act[kSegMax];
  __shared__ int s_cnt;

  const int seg = blockIdx.x;
  const Split segs(d_ff, nseg);
  const int row0 = segs.start(seg);
  const int nrows = segs.start(seg + 1) - row0;
  clear_output(y, d, meta, nseg);
  auto gate_sink = [&](int k, float s) { s_h[k] = s; };
  auto gate_row = [&](int k) { return row0 + k; };
  auto up_row = [&](int e) { return row0 + s_list[e]; };
  auto up_sink = [&](int e, float v) { seg_zval[row0 + e] = s_act[e] * (FULL ? up_value(form.silu_up, v) : v); };
  const int act = FULL ? form.act : 0;

  if constexpr (LOPA) {
    // LoPA's fixed term (G x)_i of this thread's row (written by the z kernel's extra
    // workgroups) and the squares of z for RMSNorm: loaded before the gate stream, used
    // after it, branch-free so that nothing waits for them in front of the stream
    const bool has_g = EXTRA && form.g_idx;
    const uint32_t gbits =
        EXTRA ? ldb32(make_buf(gx, 4u * (uint32_t)d_ff), has_g && (int)threadIdx.x < nrows
                                                               ? 4u * (uint32_t)(row0 + (int)threadIdx.x)
                                                               : kOOB)
              : 0u;
    const bool norm = EXTRA && form.rms_eps > 0.f;
    const int r = Cg * W::EPC;
    uint32_t sq[EXTRA ? kNormRegs : 1] = {};
    if constexpr (EXTRA) {
      const Buf qb = make_buf(zsq, 4u * (uint32_t)r);
#pragma unroll
      for (int j = 0; j < kNormRegs; ++j) {
        const int k = (int)threadIdx.x + j * kBlock;
        sq[j] = ldb32(qb, norm && k < r ? 4u * (uint32_t)k : kOOB);
      }
    }
    {
      float zr[CPLG][W::EPC];
      const int q = lane_id() & (lprg - 1);
      load_vec<W, CPLG>(z, Cg, q, lprg, zr);
      dot_rows<W, CPLG>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, zr, gate_row,
                        gate_sink);
    }
    const float gv = __builtin_bit_cast(float, gbits);
    __syncthreads();
    if constexpr (EXTRA) {
      float inv = 1.f;
      if (norm) {  // 1 / sqrt(mean z^2 + eps)
        float ss = 0.f;
#pragma unroll
        for (int j = 0; j < kNormRegs; ++j) ss += __builtin_bit_cast(float, sq[j]);
        for (int k = threadIdx.x + kNormRegs * kBlock; k < r; k += kBlock) ss += zsq[k];
        ss = wave_sum(ss);
        if (lane_id() == 0) s_ss[threadIdx.x / kWave] = ss;
        __syncthreads();
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < kBlock / kWave; ++w) tot += s_ss[w];
        inv = 1.f / sqrtf(tot / (float)r + form.rms_eps);
      }
      if (norm || form.g_idx) {  // h = inv * B (gain . z) + G x
        if ((int)threadIdx.x < nrows) s_h[threadIdx.x] = s_h[threadIdx.x] * inv + gv;
        __syncthreads();
      }
    }
    compact_segment(s_h, nrows, row0, seg, t, DENSE, act, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    float xr[CPLU][W::EPC];
    load_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU>(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  } else {
    static_assert(CPLG == CPLU, "standard gating shares the x registers");
    float xr[CPLU][W::EPC];
    load_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, xr, gate_row,
                      gate_sink);
    __syncthreads();
    compact_segment(s_h, nrows, row0, seg, t, DENSE, act, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    dot_rows<W, CPLU>(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  }
}

// y += sum over the listed neurons of a row chunk of zval * w_down_t[neuron], for one
// 64-chunk column slice (1 KB of every bf16 row, read by one wave instruction).  A
// listed neuron with zval exactly 0 (the s_gated site) is skipped: its row is not read.
// Workgroup b covers column slice b % S of the neurons in segments [c nseg/R,
// (c+1) nseg/R), c = b / S.  Its four waves take the chunk's active rows in turn;
// their partial sums are added in a fixed order and then into y with one atomic
// per column (y was cleared by the gate kernel).
template <class W, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_down_t1(const int32_t* __restrict__ seg_count,
                                                    const int32_t* __restrict__ seg_idx,
                                                    const float* __restrict__ seg_zval, int nseg, int d_ff, int R,
                                                    const uint4* __restrict__ w_down_t, int C, int d,
                                                    float* __restrict__ y) {
  constexpr int EPC = W::EPC, U = 16, kWaves = kBlock / kWave;
  extern __shared__ int s_dyn[];  // raw slots, then the compacted list (sparse only)
  __shared__ int s_cnt[kWave];
  __shared__ int s_off[kWave + 1];
  __shared__ float s_red[kWaves][kWave * EPC];

  const int S = (C + kWave - 1) / kWave;
  const int chunk = blockIdx.x / S, slice = blockIdx.x % S;
  const Split chunks(nseg, R), segs(d_ff, nseg);
  const int seg_lo = chunks.start(chunk), seg_hi = chunks.start(chunk + 1);
  const int row_lo = segs.start(seg_lo), row_hi = segs.start(seg_hi);
  const int raw_n = row_hi - row_lo;
  const int lane = lane_id(), wave = threadIdx.x / kWave;

  int n = raw_n;
  int* l_idx = nullptr;
  float* l_z = nullptr;
  if constexpr (!DENSE) {
    int* raw_idx = s_dyn;
    float* raw_z = reinterpret_cast<float*>(s_dyn + raw_n);
    l_idx = s_dyn + 2 * raw_n;
    l_z = reinterpret_cast<float*>(s_dyn + 3 * raw_n);
    // one round trip: every slot of the chunk plus the segment counts
    for (int p = threadIdx.x; p < raw_n; p += kBlock) {
      raw_idx[p] = seg_idx[row_lo + p];
      raw_z[p] = seg_zval[row_lo + p];
    }
    if (wave == 0) {
      const int nsc = seg_hi - seg_lo;  // <= 64, guaranteed by the host
      const int c = lane < nsc ? seg_count[seg_lo + lane] : 0;
      const int v = wave_inclusive_scan(c);
      s_cnt[lane] = c;
      s_off[lane] = v - c;
      if (lane == kWave - 1) s_off[kWave] = v;
    }
    __syncthreads();
    n = s_off[kWave];
    for (int p = threadIdx.x; p < raw_n; p += kBlock) {
      const int row = row_lo + p;
      const int w = segs.of(row) - seg_lo;
      const int e = row - segs.start(seg_lo + w);
      if (e < s_cnt[w]) {
        l_idx[s_off[w] + e] = raw_idx[p];
        l_z[s_off[w] + e] = raw_z[p];
      }
    }
    __syncthreads();
  }

  const int ch = slice * kWave + lane;
  const bool cvalid = ch < C;
  float acc[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
  for (int k = wave; k < n; k += kWaves * U) {
    uint4 wv[U];
    float zz[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = k + u * kWaves;
      const bool ok = kk < n;
      int row;
      if constexpr (DENSE) {
        row = row_lo + kk;
        zz[u] = ok ? seg_zval[row] : 0.f;
      } else {
        row = ok ? l_idx[kk] : 0;
        zz[u] = ok ? l_z[kk] : 0.f;
      }
      // a zero gated value (the s_gated site) needs no W_down row
      const bool need = ok && cvalid && (DENSE || zz[u] != 0.f);
      wv[u] = need ? ld_weights(w_down_t + (size_t)row * C + ch) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float f[EPC];
      unpack(W{}, wv[u], f);
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[e] = fmaf(zz[u], f[e], acc[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < EPC; ++e) s_red[wave][lane * EPC + e] = acc[e];
  __syncthreads();
  for (int o = threadIdx.x; o < kWave * EPC; o += kBlock) {
    float s = s_red[0][o];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) s += s_red[w][o];
    const int col = slice * kWave * EPC + o;
    if (col < d) unsafeAtomicAdd(y + col, s);
  }
}

// ------------------------------------------------------------------ generic kernels
// Any T <= kTokChunk, any d / d_ff / r, element-wise loads.  Used for shapes and
// batches the specialised kernels do not cover.
template <class W>
__global__ __launch_bounds__(kBlock) void k_lopa_z_generic(const float* __restrict__ x, const void* __restrict__ A,
                                                           int T, int d, int r, float* __restrict__ z) {
  const int k = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
  if (k >= r) return;
  const int lane = lane_id();
  for (int tau = 0; tau < T; ++tau) {
    float s = 0.f;
    for (int j = lane; j < d; j += kWave) s = fmaf(welem(W{}, A, (size_t)k * d + j), x[(size_t)tau * d + j], s);
    s = wave_sum(s);
    if (lane == 0) z[(size_t)tau * r + k] = s;
  }
}

template <class W, bool LOPA, bool DENSE, bool FULL>
__global__ __launch_bounds__(kBlock) void k_gate_up_generic(const float* __restrict__ x, const float* __restrict__ z,
                                                            const void* __restrict__ gate_w,
                                                            const void* __restrict__ w_up, int T, int d, int d_ff,
                                                            int r, int nseg, float t, int slots,
                                                            int32_t* __restrict__ meta,
                                                            int32_t* __restrict__ seg_count,
                                                            int32_t* __restrict__ seg_idx,
                                                            float* __restrict__ seg_act,
                                                            float* __restrict__ seg_zval, float* __restrict__ y,
                                                            Form form) {
  __shared__ float s_h[kSegMax][kTokChunk];
  __shared__ int s_list[kSegMax];
  __shared__ int s_cnt;
  const int seg = blockIdx.x;
  const Split segs(d_ff, nseg);
  const int row0 = segs.start(seg), nrows = segs.start(seg + 1) - row0;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  constexpr int kWaves = kBlock / kWave;
  const int len = LOPA ? r : d;
  const float* vec = LOPA ? z : x;
  clear_output(y, T * d, meta, nseg);

  for (int k = wave; k < nrows; k += kWaves) {
    const size_t rowoff = (size_t)(row0 + k) * len;
    for (int tau = 0; tau < T; ++tau) {
      float s = 0.f;
      for (int j = lane; j < len; j += kWave) s = fmaf(welem(W{}, gate_w, rowoff + j), vec[(size_t)tau * len + j], s);
      s = wave_sum(s);
      if (lane == 0) s_h[k][tau] = s;
    }
  }
  __syncthreads();
  if constexpr (FULL) {
    if (form.g_idx) {  // LoPA's fixed term: h += G x
      for (int o = threadIdx.x; o < nrows * T; o += kBlock) {
        const int k = o / T, tau = o - k * T;
        s_h[k][tau] += g_gather(g_fetch(form, d_ff, row0 + k), x + (size_t)tau * d, d);
      }
      __syncthreads();
    }
  }

  if (threadIdx.x < kWave) {
    const bool valid = lane < nrows;
    bool any = false;
    if (valid)
      for (int tau = 0; tau < T; ++tau) any |= s_h[lane][tau] > t;
    const bool sel = valid && (DENSE || any);
    const uint64_t m = __ballot(sel);
    const int rank = rank_in_mask(m);
    if (sel) {
      s_list[rank] = lane;
      seg_idx[row0 + rank] = row0 + lane;
      for (int tau = 0; tau < T; ++tau) {
        const float h = s_h[lane][tau];
        const float a = h > t ? (FULL ? gate_value(form.act, h - t) : h - t) : 0.f;
        s_h[lane][tau] = a;  // this lane owns row `lane`: overwrite h with the activation
        seg_act[(size_t)tau * slots + row0 + rank] = a;
      }
    }
    if (lane == 0) {
      s_cnt = __popcll(m);
      seg_count[seg] = s_cnt;
    }
  }
  __syncthreads();

  const int cnt = s_cnt;
  for (int e = wave; e < cnt; e += kWaves) {
    const int kr = s_list[e];
    const size_t rowoff = (size_t)(row0 + kr) * d;
    for (int tau = 0; tau < T; ++tau) {
      float s = 0.f;
      for (int j = lane; j < d; j += kWave) s = fmaf(welem(W{}, w_up, rowoff + j), x[(size_t)tau * d + j], s);
      s = wave_sum(s);
      if (lane == 0) seg_zval[(size_t)tau * slots + row0 + e] = s_h[kr][tau] * (FULL ? up_value(form.silu_up, s) : s);
    }
  }
}

// thread per output column; tokens in groups of 8 accumulators; y written directly
template <class W, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_down_generic(const int32_t* __restrict__ seg_count,
                                                         const int32_t* __restrict__ seg_idx,
                                                         const float* __restrict__ seg_zval, int nseg, int d_ff,
                                                         int slots, const void* __restrict__ w_down_t, int T, int d,
                                                         float* __restrict__ y) {
  extern __shared__ int s_pre[];  // [nseg + 1] list offsets (sparse only)
  __shared__ int s_slot[kListWindow];
  const int col = blockIdx.x * kBlock + threadIdx.x;
  const bool cvalid = col < d;
  int n = d_ff;
  if (!DENSE) {
    for (int s = threadIdx.x; s < nseg; s += kBlock) s_pre[s] = seg_count[s];
    __syncthreads();
    block_exclusive_scan(s_pre, nseg);
    n = s_pre[nseg];
  }
  for (int tg = 0; tg < T; tg += 8) {
    const int tn = min(8, T - tg);
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.f;
    for (int base = 0; base < n; base += kListWindow) {
      const int wn = min(kListWindow, n - base);
      if (!DENSE) {
        const Split segs(d_ff, nseg);
        for (int s = threadIdx.x; s < nseg; s += kBlock) {
          const int k0 = s_pre[s], k1 = s_pre[s + 1];
          const int lo = max(k0, base), hi = min(k1, base + wn);
          const int slot0 = segs.start(s);
          for (int k = lo; k < hi; ++k) s_slot[k - base] = slot0 + (k - k0);
        }
        __syncthreads();
      }
      if (cvalid) {
        for (int k = 0; k < wn; ++k) {
          const int slot = DENSE ? base + k : s_slot[k];
          const int row = DENSE ? slot : seg_idx[slot];
          const float w = welem(W{}, w_down_t, (size_t)row * d + col);
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (u < tn) {
              const float zv = seg_zval[(size_t)(tg + u) * slots + slot];
              if (DENSE || zv != 0.f) acc[u] = fmaf(zv, w, acc[u]);  // s_gated: zero adds nothing
            }
        }
      }
      if (!DENSE) __syncthreads();
    }
    if (cvalid)
      for (int u = 0; u < tn; ++u) y[(size_t)(tg + u) * d + col] = acc[u];
  }
}

// ------------------------------------------------------------------ launch helpers
int ilog2(int v) {
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

// lanes per row for a row of C chunks so that each lane holds at most `cpl` chunks
int lanes_per_row(int C, int cpl) {
  int lpr = 1;
  while (lpr < kWave && lpr * cpl < C) lpr <<= 1;
  return lpr;
}

int cpl_for(int C) { return C <= 8 * kWave ? 8 : (C <= 16 * kWave ? 16 : 0); }

int cu_count() {
  static int cus[16] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  const int slot = dev & 15;
  if (cus[slot] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[slot] = n;
  }
  return cus[slot];
}

// Segments for the T = 1 gate kernel: one row-balanced segment per workgroup slot the
// GPU holds at once (so every CU gets the same number of rows; more segments than
// resident slots measured slower), never more than kSegMax rows per segment.  `per_cu`
// caches the kernel's occupancy.
template <class K>
int resident_segments(K kernel, int* per_cu, int d_ff) {
  if (*per_cu == 0) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, 0) != hipSuccess || n <= 0) n = 1;
    *per_cu = n;
  }
  int g = cu_count() * *per_cu;
  const int lo = (d_ff + kSegMax - 1) / kSegMax;
  if (g < lo) g = lo;
  if (g > d_ff) g = d_ff;
  return g;
}

// The fast single-token kernels address a matrix with 32-bit byte offsets below 2^31.
bool fast_ok(const Shape& sh, Gate g) {
  const int epc_ = sh.wdt == 1 ? WBf16::EPC : WF32::EPC;
  const int64_t wb = sh.wdt == 1 ? 2 : 4, lim = int64_t(1) << 31;
  if (sh.T != 1 || sh.d % epc_ != 0 || cpl_for(sh.d / epc_) == 0) return false;
  if (wb * sh.d_ff * sh.d >= lim) return false;
  if (g == Gate::LoPA && (sh.r % epc_ != 0 || cpl_for(sh.r / epc_) == 0 || wb * sh.r * sh.d >= lim ||
                          wb * sh.d_ff * sh.r >= lim))
    return false;
  return true;
}

template <class W, bool LOPA, bool DENSE, int FORM, int CPLG, int CPLU>
hipError_t go_gate_up_t1(const Shape& sh, const Form& form, const float* x, const void* gate_w, const void* w_up,
                         float t, Workspace& ws, float* y, hipStream_t s) {
  const int Cu = sh.d / W::EPC, Cg = LOPA ? sh.r / W::EPC : Cu;
  const int lpru = lanes_per_row(Cu, CPLU), lprg = lanes_per_row(Cg, CPLG);
  auto kernel = k_gate_up_t1<W, LOPA, DENSE, CPLG, CPLU, FORM>;
  static int per_cu = 0;  // one cache per instantiation
  ws.nseg = resident_segments(kernel, &per_cu, sh.d_ff);
  return launch_gate_kernel(kernel, ws.nseg, s, x, (const float*)ws.z, static_cast<const uint4*>(gate_w), Cg, lprg,
                            ilog2(lprg), static_cast<const uint4*>(w_up), Cu, lpru, ilog2(lpru), sh.d_ff, ws.nseg, t,
                            ws.meta, ws.seg_count, ws.seg_idx, ws.seg_act, ws.seg_zval, y, sh.d, form,
                            (const float*)ws.zsq, (const float*)ws.gx);
}

template <class W, bool LOPA, bool DENSE, int FORM>
hipError_t gate_up_fast(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up, float t,
                        Workspace& ws, float* y, hipStream_t s) {
  const int cplu = cpl_for(sh.d / W::EPC);
  if constexpr (LOPA) {
    const int cplg = cpl_for(sh.r / W::EPC);
    if (cplg == 8 && cplu == 8) return go_gate_up_t1<W, true, DENSE, FORM, 8, 8>(sh, f, x, gate_w, w_up, t, ws, y, s);
    if (cplg == 8 && cplu == 16)
      return go_gate_up_t1<W, true, DENSE, FORM, 8, 16>(sh, f, x, gate_w, w_up, t, ws, y, s);
    if (cplg == 16 && cplu == 8)
      return go_gate_up_t1<W, true, DENSE, FORM, 16, 8>(sh, f, x, gate_w, w_up, t, ws, y, s);
    return go_gate_up_t1<W, true, DENSE, FORM, 16, 16>(sh, f, x, gate_w, w_up, t, ws, y, s);
  } else {
    if (cplu == 8) return go_gate_up_t1<W, false, DENSE, FORM, 8, 8>(sh, f, x, gate_w, w_up, t, ws, y, s);
    return go_gate_up_t1<W, false, DENSE, FORM, 16, 16>(sh, f, x, gate_w, w_up, t, ws, y, s);
  }
}

template <class W, bool LOPA, bool DENSE, bool FULL>
hipError_t gate_up_generic(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up,
                           float t, Workspace& ws, float* y, hipStream_t s) {
  ws.nseg = (sh.d_ff + kSegGeneric - 1) / kSegGeneric;
  return launch_gate_kernel(k_gate_up_generic<W, LOPA, DENSE, FULL>, ws.nseg, s, x, (const float*)ws.z, gate_w, w_up,
                            sh.T, sh.d, sh.d_ff, sh.r, ws.nseg, t, ws.slots, ws.meta, ws.seg_count, ws.seg_idx,
                            ws.seg_act, ws.seg_zval, y, f);
}

// RMSNorm on z (Section 3.3), one workgroup per token: the partial copies summed into
// copy 0 and scaled by gain / sqrt(mean z^2 + eps); the other copies zeroed.  The first
// kNormRegs * kBlock components stay in registers between the two passes.
__global__ __launch_bounds__(kBlock) void k_rms_norm(float* __restrict__ z, int parts, int tc, int r,
                                                     const float* __restrict__ gain, float eps) {
  __shared__ float s_part[kBlock / kWave];
  const int tok = blockIdx.x;
  auto zsum = [&](int k) {
    float v = 0.f;
    for (int p = 0; p < parts; ++p) v += z[((size_t)p * tc + tok) * r + k];
    return v;
  };
  float v[kNormRegs];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kNormRegs; ++j) {
    const int k = (int)threadIdx.x + j * kBlock;
    v[j] = k < r ? zsum(k) : 0.f;
    ss = fmaf(v[j], v[j], ss);
  }
  for (int k = threadIdx.x + kNormRegs * kBlock; k < r; k += kBlock) {
    const float u = zsum(k);
    ss = fmaf(u, u, ss);
  }
  ss = wave_sum(ss);
  if (lane_id() == 0) s_part[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kBlock / kWave; ++w) tot += s_part[w];
  const float inv = 1.f / sqrtf(tot / (float)r + eps);
  auto put = [&](int k, float u) {
    z[(size_t)tok * r + k] = u * inv * (gain ? gain[k] : 1.f);
    for (int p = 1; p < parts; ++p) z[((size_t)p * tc + tok) * r + k] = 0.f;
  };
  for (int k = threadIdx.x + kNormRegs * kBlock; k < r; k += kBlock) put(k, zsum(k));
#pragma unroll
  for (int j = 0; j < kNormRegs; ++j) {
    const int k = (int)threadIdx.x + j * kBlock;
    if (k < r) put(k, v[j]);
  }
}

template <class W>
hipError_t lopa_z(const Shape& sh, const Form& form, const float* x, const void* A, const Workspace& ws,
                  hipStream_t s) {
  if (fast_ok(sh, Gate::LoPA)) {
    const int C = sh.d / W::EPC;
    const int cpl = cpl_for(C), lpr = lanes_per_row(C, cpl), lg = ilog2(lpr);
    const int rows_per_block = (kBlock / kWave) * (kWave >> lg);
    const int grid = (sh.r + rows_per_block - 1) / rows_per_block;
    const uint4* a = static_cast<const uint4*>(A);
    const bool norm = form.rms_eps > 0.f;
    // with G, extra workgroups write G x for the gate kernel
    const GWork gw{form, x, ws.gx, 1, sh.d, sh.d_ff, grid};
    const int g = grid + (form.g_idx ? (g_items(sh.d_ff, 1) + kBlock - 1) / kBlock : 0);
    if (cpl == 8 && norm)
      k_lopa_z_t1<W, 8, true><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, form.rms_gain, ws.zsq, gw);
    else if (cpl == 8)
      k_lopa_z_t1<W, 8, false><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, nullptr, nullptr, gw);
    else if (norm)
      k_lopa_z_t1<W, 16, true><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, form.rms_gain, ws.zsq, gw);
    else
      k_lopa_z_t1<W, 16, false><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, nullptr, nullptr, gw);
  } else {
    const int grid = (sh.r + kBlock / kWave - 1) / (kBlock / kWave);
    k_lopa_z_generic<W><<<grid, kBlock, 0, s>>>(x, A, sh.T, sh.d, sh.r, ws.z);
  }
  return hipGetLastError();
}

// Down-projection grid for T = 1: S column slices x R row chunks, about
// kDownWgPerCu workgroups per CU, at most 64 segments per chunk.
constexpr int kDownWgPerCu = 2;

void down_grid(int C, int nseg, int d_ff, int* S, int* R, size_t* shmem_rows) {
  *S = (C + kWave - 1) / kWave;
  int r = (kDownWgPerCu * cu_count() + *S - 1) / *S;
  const int rmin = (nseg + kWave - 1) / kWave;
  if (r < rmin) r = rmin;
  if (r > nseg) r = nseg;
  *R = r;
  // largest row range of a chunk: ceil(nseg / R) segments of at most ceil(d_ff / nseg) rows
  *shmem_rows = (size_t)((nseg + r - 1) / r) * (size_t)((d_ff + nseg - 1) / nseg);
}

template <class W, bool DENSE>
hipError_t down(const Shape& sh, const void* w_down_t, const Workspace& ws, float* y, hipStream_t s) {
  if (sh.T == 1 && sh.d % W::EPC == 0) {
    const int C = sh.d / W::EPC;
    int S, R;
    size_t rows;
    down_grid(C, ws.nseg, sh.d_ff, &S, &R, &rows);
    const size_t shmem = DENSE ? 0 : 4 * sizeof(int) * rows;
    if (shmem > 96 * 1024) return hipErrorInvalidValue;
    k_down_t1<W, DENSE><<<S * R, kBlock, shmem, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff, R,
                                                      static_cast<const uint4*>(w_down_t), C, sh.d, y);
  } else {
    const size_t shmem = DENSE ? 0 : sizeof(int) * (size_t)(ws.nseg + 1);
    const int grid = (sh.d + kBlock - 1) / kBlock;
    k_down_generic<W, DENSE><<<grid, kBlock, shmem, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff,
                                                        ws.slots, w_down_t, sh.T, sh.d, y);
  }
  return hipGetLastError();
}

// the kernels for the form: the compile-time kind of the single-token kernel, the full
// flag of the element-wise one (G and the norm need LoPA; the options check enforces it)
template <class W, bool LOPA, bool DENSE>
hipError_t gate_up_form(const Shape& sh, bool fast, const Form& f, const float* x, const void* gate_w,
                        const void* w_up, float t, Workspace& ws, float* y, hipStream_t s) {
  if (!fast)
    return f.full() ? gate_up_generic<W, LOPA, DENSE, true>(sh, f, x, gate_w, w_up, t, ws, y, s)
                    : gate_up_generic<W, LOPA, DENSE, false>(sh, f, x, gate_w, w_up, t, ws, y, s);
  if constexpr (LOPA)
    if (f.kind() == kFormLoPA) return gate_up_fast<W, LOPA, DENSE, kFormLoPA>(sh, f, x, gate_w, w_up, t, ws, y, s);
  return f.full() ? gate_up_fast<W, LOPA, DENSE, kFormAct>(sh, f, x, gate_w, w_up, t, ws, y, s)
                  : gate_up_fast<W, LOPA, DENSE, kFormDefault>(sh, f, x, gate_w, w_up, t, ws, y, s);
}

}  // namespace

// ------------------------------------------------------------------ launchers
hipError_t launch_rms_norm(float* z, int parts, int tc, int T, int r, const float* gain, float eps, hipStream_t s) {
  k_rms_norm<<<T, kBlock, 0, s>>>(z, parts, tc, r, gain, eps);
  return hipGetLastError();
}

hipError_t launch_lopa_z(const Shape& sh, const Form& form, const float* x, const void* lopa_a, const Workspace& ws,
                         hipStream_t s) {
  return sh.wdt == 1 ? lopa_z<WBf16>(sh, form, x, lopa_a, ws, s) : lopa_z<WF32>(sh, form, x, lopa_a, ws, s);
}

hipError_t launch_gate_up(const Shape& sh, Gate g, bool dense, const Form& form, const float* x, const void* gate_w,
                          const void* w_up, float t, Workspace& ws, float* y, hipStream_t s) {
  const bool lopa = g == Gate::LoPA;
  const bool fast = fast_ok(sh, g);
  if (lopa && !fast && form.rms_eps > 0.f) {  // the single-token kernel normalises z itself
    const hipError_t e = launch_rms_norm(ws.z, 1, ws.tc, sh.T, sh.r, form.rms_gain, form.rms_eps, s);
    if (e != hipSuccess) return e;
  }
  if (sh.wdt == 1) {
    if (lopa) return dense ? gate_up_form<WBf16, true, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s)
                           : gate_up_form<WBf16, true, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s);
    return dense ? gate_up_form<WBf16, false, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s)
                 : gate_up_form<WBf16, false, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s);
  }
  if (lopa) return dense ? gate_up_form<WF32, true, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s)
                         : gate_up_form<WF32, true, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s);
  return dense ? gate_up_form<WF32, false, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s)
               : gate_up_form<WF32, false, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s);
}

hipError_t launch_down(const Shape& sh, bool dense, const void* w_down_t, const Workspace& ws, float* y,
                       hipStream_t s) {
  if (sh.wdt == 1)
    return dense ? down<WBf16, true>(sh, w_down_t, ws, y, s) : down<WBf16, false>(sh, w_down_t, ws, y, s);
  return dense ? down<WF32, true>(sh, w_down_t, ws, y, s) : down<WF32, false>(sh, w_down_t, ws, y, s);
}

}  // namespace ffn

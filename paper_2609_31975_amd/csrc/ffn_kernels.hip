// gfx950 kernels of the activation-sparse FFN forward pass.
//
// Data flow of one pass (paper Section 3.1: the gate is computed in full, zeros of
// A(W1 x) are known before W3 and W2 are touched; Section 3.3: LoPA gate B (A x)):
//
//   [LoPA only] k_lopa_z*     z = A x                               -> ws.z
//   k_gate_up*                per workgroup = one segment of kSeg consecutive
//                             neurons: h = W_gate x (or B z), ballot compaction of
//                             the neurons with h > t (union over tokens), then the
//                             W_up row dot products of exactly those neurons:
//                             act = h - t, zval = act * <w_up[i], x>
//                             -> seg_count / seg_idx / seg_act / seg_zval
//   k_down*                   y = sum_k zval_k * w_down_t[idx_k], each workgroup
//                             owning a 16-column slice of y for all active rows;
//                             prefix sums of seg_count give the ascending list.
//
// No atomics and no inter-workgroup waits: every output element is written by one
// thread after a fixed-order reduction, so results are bit-reproducible.
#include "ffn_internal.h"

namespace ffn {
namespace {

// ------------------------------------------------------------------ weight formats
struct WBf16 {
  static constexpr int EPC = 8;  // elements per 16-byte chunk
};
struct WF32 {
  static constexpr int EPC = 4;
};

__device__ __forceinline__ void unpack(WBf16, const uint4& v, float (&f)[8]) {
  // a bf16 is the high half of an fp32: shift the low element up, mask the high one
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xffff0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xffff0000u);
  f[4] = __uint_as_float(v.z << 16);
  f[5] = __uint_as_float(v.z & 0xffff0000u);
  f[6] = __uint_as_float(v.w << 16);
  f[7] = __uint_as_float(v.w & 0xffff0000u);
}
__device__ __forceinline__ void unpack(WF32, const uint4& v, float (&f)[4]) {
  f[0] = __uint_as_float(v.x);
  f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z);
  f[3] = __uint_as_float(v.w);
}

__device__ __forceinline__ float welem(WBf16, const void* w, size_t k) {
  return __uint_as_float((uint32_t)(static_cast<const uint16_t*>(w)[k]) << 16);
}
__device__ __forceinline__ float welem(WF32, const void* w, size_t k) {
  return static_cast<const float*>(w)[k];
}

// Weights are read once per call: stream them past the caches.
__device__ __forceinline__ uint4 ld_weights(const uint4* p) {
  typedef unsigned u4v __attribute__((ext_vector_type(4)));
  u4v t = __builtin_nontemporal_load(reinterpret_cast<const u4v*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// sum over aligned groups of `width` lanes (width a power of two <= 64)
__device__ __forceinline__ float group_sum(float v, int width) {
  for (int o = width >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_sum(float v) { return group_sum(v, kWave); }

__device__ __forceinline__ int rank_in_mask(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

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

template <int CPL>
__device__ __forceinline__ void load_row(const uint4* __restrict__ row, bool valid, int C, int q, int lpr,
                                         uint4 (&b)[CPL]) {
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = q + c * lpr;
    b[c] = (valid && ch < C) ? ld_weights(row + ch) : make_uint4(0u, 0u, 0u, 0u);
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

// Dot products <rows, v> for rows picked by `row_of(k)`, k in [0, n): waves take
// passes of 64/lpr rows, two passes in flight; `sink(k, value)` runs on lane q == 0.
template <class W, int CPL, class RowOf, class Sink>
__device__ __forceinline__ void dot_rows(const uint4* __restrict__ mat, int C, int lpr, int lpr_log2, int n,
                                         const float (&v)[CPL][W::EPC], RowOf row_of, Sink sink) {
  constexpr int kWaves = kBlock / kWave;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int q = lane & (lpr - 1), p = lane >> lpr_log2;
  const int rpp = kWave >> lpr_log2;
  const int npass = (n + rpp - 1) / rpp;
  for (int pass = wave; pass < npass; pass += 2 * kWaves) {
    const int k0 = pass * rpp + p;
    const int k1 = (pass + kWaves) * rpp + p;
    const bool v0 = k0 < n, v1 = k1 < n;
    uint4 b0[CPL], b1[CPL];
    load_row<CPL>(mat + (size_t)row_of(v0 ? k0 : 0) * C, v0, C, q, lpr, b0);
    load_row<CPL>(mat + (size_t)row_of(v1 ? k1 : 0) * C, v1, C, q, lpr, b1);
    const float s0 = group_sum(lane_dot<W, CPL>(b0, v), lpr);
    const float s1 = group_sum(lane_dot<W, CPL>(b1, v), lpr);
    if (q == 0) {
      if (v0) sink(k0, s0);
      if (v1) sink(k1, s1);
    }
  }
}

// ------------------------------------------------------------------ fast kernels, T = 1
// z = A x for one token (rows of A: C chunks).
template <class W, int CPL>
__global__ __launch_bounds__(kBlock) void k_lopa_z_t1(const float* __restrict__ x, const uint4* __restrict__ A,
                                                      int C, int lpr, int lpr_log2, int r, float* __restrict__ z) {
  float xr[CPL][W::EPC];
  load_vec<W, CPL>(x, C, lane_id() & (lpr - 1), lpr, xr);
  const int rows_per_block = (kBlock / kWave) * 2 * (kWave >> lpr_log2);
  const int k0 = blockIdx.x * rows_per_block;
  const int n = min(rows_per_block, r - k0);
  dot_rows<W, CPL>(A, C, lpr, lpr_log2, n, xr, [&](int k) { return k0 + k; },
                   [&](int k, float s) { z[k0 + k] = s; });
}

// Ballot compaction of one segment (run by the first wave): neurons whose gate value
// exceeds t (all neurons if `all`) get ascending ranks; their activation h - t is
// kept in LDS for the W_up phase and published with the neuron index.
__device__ __forceinline__ void compact_segment(const float* s_h, int nrows, int row0, int seg, float t, bool all,
                                                int* s_list, float* s_act, int* s_cnt, int32_t* seg_count,
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
      const float a = on ? h - t : 0.f;
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

// One segment of kSeg neurons: gate, compaction, W_up dots of the selected neurons.
// LOPA: the gate rows are B [d_ff][r] against z; otherwise W_gate [d_ff][d] against x.
// DENSE: every neuron of the segment is selected (act = max(h - t, 0)).
template <class W, bool LOPA, bool DENSE, int CPLG, int CPLU>
__global__ __launch_bounds__(kBlock) void k_gate_up_t1(const float* __restrict__ x, const float* __restrict__ z,
                                                       const uint4* __restrict__ gate_w, int Cg, int lprg,
                                                       int lprg_log2, const uint4* __restrict__ w_up, int Cu,
                                                       int lpru, int lpru_log2, int d_ff, float t,
                                                       int32_t* __restrict__ seg_count,
                                                       int32_t* __restrict__ seg_idx, float* __restrict__ seg_act,
                                                       float* __restrict__ seg_zval) {
  __shared__ float s_h[kSeg];
  __shared__ int s_list[kSeg];
  __shared__ float s_act[kSeg];
  __shared__ int s_cnt;

  const int seg = blockIdx.x;
  const int row0 = seg * kSeg;
  const int nrows = min(kSeg, d_ff - row0);
  auto gate_sink = [&](int k, float s) { s_h[k] = s; };
  auto gate_row = [&](int k) { return row0 + k; };
  auto up_row = [&](int e) { return row0 + s_list[e]; };
  auto up_sink = [&](int e, float v) { seg_zval[row0 + e] = s_act[e] * v; };

  if constexpr (LOPA) {
    {
      float zr[CPLG][W::EPC];
      load_vec<W, CPLG>(z, Cg, lane_id() & (lprg - 1), lprg, zr);
      dot_rows<W, CPLG>(gate_w, Cg, lprg, lprg_log2, nrows, zr, gate_row, gate_sink);
    }
    __syncthreads();
    compact_segment(s_h, nrows, row0, seg, t, DENSE, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    float xr[CPLU][W::EPC];
    load_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU>(w_up, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  } else {
    static_assert(CPLG == CPLU, "standard gating shares the x registers");
    float xr[CPLU][W::EPC];
    load_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU>(gate_w, Cg, lprg, lprg_log2, nrows, xr, gate_row, gate_sink);
    __syncthreads();
    compact_segment(s_h, nrows, row0, seg, t, DENSE, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    dot_rows<W, CPLU>(w_up, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  }
}

// ------------------------------------------------------------------ down projection
// Exclusive prefix sum of s[0..n) in place, s[n] = total; all kBlock threads call it.
__device__ void block_exclusive_scan(int* s, int n) {
  __shared__ int s_wsum[kBlock / kWave];
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int per = (n + kBlock - 1) / kBlock;
  const int b = min((int)threadIdx.x * per, n), e = min(b + per, n);
  int local = 0;
  for (int i = b; i < e; ++i) local += s[i];
  int v = local;
  for (int o = 1; o < kWave; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  if (lane == kWave - 1) s_wsum[wave] = v;
  __syncthreads();
  int excl = v - local;
  for (int w = 0; w < wave; ++w) excl += s_wsum[w];
  for (int i = b; i < e; ++i) {
    const int c = s[i];
    s[i] = excl;
    excl += c;
  }
  if (threadIdx.x == kBlock - 1) s[n] = excl;
  __syncthreads();
}

// Load segment counts and turn them into ascending-list offsets; returns the total.
__device__ int segment_offsets(const int32_t* __restrict__ seg_count, int nseg, int* s_pre) {
  for (int s = threadIdx.x; s < nseg; s += kBlock) s_pre[s] = seg_count[s];
  __syncthreads();
  block_exclusive_scan(s_pre, nseg);
  return s_pre[nseg];
}

// Stage list entries [base, base + wn) into LDS as slot numbers.
__device__ void stage_window(const int* s_pre, int nseg, int base, int wn, int* s_slot) {
  for (int s = threadIdx.x; s < nseg; s += kBlock) {
    const int k0 = s_pre[s], k1 = s_pre[s + 1];
    const int lo = max(k0, base), hi = min(k1, base + wn);
    for (int k = lo; k < hi; ++k) s_slot[k - base] = s * kSeg + (k - k0);
  }
}

// Map workgroup -> column slice so that neighbouring slices (which share 128-byte
// lines of each weight row) run on the same XCD: workgroups are dealt round-robin
// over the 8 XCDs, so group b % 8 gets a contiguous range of slices.
__device__ __forceinline__ int xcd_slice(int b, int nslices) {
  return (nslices % 8 == 0) ? (b % 8) * (nslices / 8) + b / 8 : b;
}

// y (one token) = sum over listed neurons of zval * w_down_t[row]; the workgroup owns
// CPW chunks (16 columns) of y and reduces its row groups in a fixed order.
template <class W, int CPW, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_down_t1(const int32_t* __restrict__ seg_count,
                                                    const int32_t* __restrict__ seg_idx,
                                                    const float* __restrict__ seg_zval, int nseg, int d_ff,
                                                    const uint4* __restrict__ w_down_t, int C, int d,
                                                    float* __restrict__ y) {
  extern __shared__ int s_pre[];  // [nseg + 1]
  __shared__ int s_slot[kListWindow];
  constexpr int EPC = W::EPC, NRG = kBlock / CPW, OUT = CPW * EPC, NB = kBlock / OUT;
  __shared__ float s_red[kBlock * EPC];
  __shared__ float s_red2[kBlock];
  constexpr int U = 8;

  const int nslices = (C + CPW - 1) / CPW;
  const int slice = xcd_slice(blockIdx.x, nslices);
  const int cc = threadIdx.x % CPW, rg = threadIdx.x / CPW;
  const int ch = slice * CPW + cc;
  const bool cvalid = ch < C;

  float acc[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) acc[e] = 0.f;

  const int n = DENSE ? d_ff : segment_offsets(seg_count, nseg, s_pre);
  for (int base = 0; base < n; base += kListWindow) {
    const int wn = min(kListWindow, n - base);
    if (!DENSE) {
      stage_window(s_pre, nseg, base, wn, s_slot);
      __syncthreads();
    }
    for (int k = rg; k < wn; k += NRG * U) {
      uint4 wv[U];
      float zz[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kk = k + u * NRG;
        const bool ok = kk < wn;
        const int slot = ok ? (DENSE ? base + kk : s_slot[kk]) : 0;
        const int row = DENSE ? slot : (ok ? seg_idx[slot] : 0);
        zz[u] = ok ? seg_zval[slot] : 0.f;
        wv[u] = (ok && cvalid) ? ld_weights(w_down_t + (size_t)row * C + ch) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float f[EPC];
        unpack(W{}, wv[u], f);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] = fmaf(zz[u], f[e], acc[e]);
      }
    }
    if (!DENSE) __syncthreads();
  }

  // fixed-order reduction over the NRG row groups: [rg][cc][e] -> NB partials -> 1
#pragma unroll
  for (int e = 0; e < EPC; ++e) s_red[(rg * CPW + cc) * EPC + e] = acc[e];
  __syncthreads();
  {
    const int o = threadIdx.x % OUT, blk = threadIdx.x / OUT;
    constexpr int PER = NRG / NB;
    float s = 0.f;
    for (int g = blk * PER; g < (blk + 1) * PER; ++g) s += s_red[g * OUT + o];
    s_red2[blk * OUT + o] = s;
  }
  __syncthreads();
  if (threadIdx.x < OUT) {
    float s = 0.f;
    for (int b2 = 0; b2 < NB; ++b2) s += s_red2[b2 * OUT + threadIdx.x];
    const int col = slice * OUT + threadIdx.x;
    if (col < d) y[col] = s;
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

template <class W, bool LOPA, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_gate_up_generic(const float* __restrict__ x, const float* __restrict__ z,
                                                            const void* __restrict__ gate_w,
                                                            const void* __restrict__ w_up, int T, int d, int d_ff,
                                                            int r, float t, int slots, int32_t* __restrict__ seg_count,
                                                            int32_t* __restrict__ seg_idx,
                                                            float* __restrict__ seg_act,
                                                            float* __restrict__ seg_zval) {
  __shared__ float s_h[kSeg][kTokChunk];
  __shared__ int s_list[kSeg];
  __shared__ int s_cnt;
  const int seg = blockIdx.x, row0 = seg * kSeg, nrows = min(kSeg, d_ff - row0);
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  constexpr int kWaves = kBlock / kWave;
  const int len = LOPA ? r : d;
  const float* vec = LOPA ? z : x;

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
        const float a = h > t ? h - t : 0.f;
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
      if (lane == 0) seg_zval[(size_t)tau * slots + row0 + e] = s_h[kr][tau] * s;
    }
  }
}

// thread per output column; tokens in groups of 8 accumulators
template <class W, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_down_generic(const int32_t* __restrict__ seg_count,
                                                         const int32_t* __restrict__ seg_idx,
                                                         const float* __restrict__ seg_zval, int nseg, int d_ff,
                                                         int slots, const void* __restrict__ w_down_t, int T, int d,
                                                         float* __restrict__ y) {
  extern __shared__ int s_pre[];
  __shared__ int s_slot[kListWindow];
  const int col = blockIdx.x * kBlock + threadIdx.x;
  const bool cvalid = col < d;
  const int n = DENSE ? d_ff : segment_offsets(seg_count, nseg, s_pre);
  for (int tg = 0; tg < T; tg += 8) {
    const int tn = min(8, T - tg);
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.f;
    for (int base = 0; base < n; base += kListWindow) {
      const int wn = min(kListWindow, n - base);
      if (!DENSE) {
        stage_window(s_pre, nseg, base, wn, s_slot);
        __syncthreads();
      }
      if (cvalid) {
        for (int k = 0; k < wn; ++k) {
          const int slot = DENSE ? base + k : s_slot[k];
          const int row = DENSE ? slot : seg_idx[slot];
          const float w = welem(W{}, w_down_t, (size_t)row * d + col);
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (u < tn) acc[u] = fmaf(seg_zval[(size_t)(tg + u) * slots + slot], w, acc[u]);
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

bool fast_ok(const Shape& sh, Gate g) {
  const int epc_ = sh.wdt == 1 ? WBf16::EPC : WF32::EPC;
  if (sh.T != 1 || sh.d % epc_ != 0 || cpl_for(sh.d / epc_) == 0) return false;
  if (g == Gate::LoPA && (sh.r % epc_ != 0 || cpl_for(sh.r / epc_) == 0)) return false;
  return true;
}

template <class W, bool LOPA, bool DENSE, int CPLG, int CPLU>
hipError_t go_gate_up_t1(const Shape& sh, const float* x, const void* gate_w, const void* w_up, float t,
                         const Workspace& ws, hipStream_t s) {
  const int Cu = sh.d / W::EPC, Cg = LOPA ? sh.r / W::EPC : Cu;
  const int lpru = lanes_per_row(Cu, CPLU), lprg = lanes_per_row(Cg, CPLG);
  k_gate_up_t1<W, LOPA, DENSE, CPLG, CPLU><<<ws.nseg, kBlock, 0, s>>>(
      x, ws.z, static_cast<const uint4*>(gate_w), Cg, lprg, ilog2(lprg), static_cast<const uint4*>(w_up), Cu, lpru,
      ilog2(lpru), sh.d_ff, t, ws.seg_count, ws.seg_idx, ws.seg_act, ws.seg_zval);
  return hipGetLastError();
}

template <class W, bool LOPA, bool DENSE>
hipError_t gate_up_fast(const Shape& sh, const float* x, const void* gate_w, const void* w_up, float t,
                        const Workspace& ws, hipStream_t s) {
  const int cplu = cpl_for(sh.d / W::EPC);
  if constexpr (LOPA) {
    const int cplg = cpl_for(sh.r / W::EPC);
    if (cplg == 8 && cplu == 8) return go_gate_up_t1<W, true, DENSE, 8, 8>(sh, x, gate_w, w_up, t, ws, s);
    if (cplg == 8 && cplu == 16) return go_gate_up_t1<W, true, DENSE, 8, 16>(sh, x, gate_w, w_up, t, ws, s);
    if (cplg == 16 && cplu == 8) return go_gate_up_t1<W, true, DENSE, 16, 8>(sh, x, gate_w, w_up, t, ws, s);
    return go_gate_up_t1<W, true, DENSE, 16, 16>(sh, x, gate_w, w_up, t, ws, s);
  } else {
    if (cplu == 8) return go_gate_up_t1<W, false, DENSE, 8, 8>(sh, x, gate_w, w_up, t, ws, s);
    return go_gate_up_t1<W, false, DENSE, 16, 16>(sh, x, gate_w, w_up, t, ws, s);
  }
}

template <class W, bool LOPA, bool DENSE>
hipError_t gate_up_generic(const Shape& sh, const float* x, const void* gate_w, const void* w_up, float t,
                           const Workspace& ws, hipStream_t s) {
  k_gate_up_generic<W, LOPA, DENSE><<<ws.nseg, kBlock, 0, s>>>(x, ws.z, gate_w, w_up, sh.T, sh.d, sh.d_ff, sh.r, t,
                                                               ws.slots, ws.seg_count, ws.seg_idx, ws.seg_act,
                                                               ws.seg_zval);
  return hipGetLastError();
}

template <class W>
hipError_t lopa_z(const Shape& sh, const float* x, const void* A, const Workspace& ws, hipStream_t s) {
  if (fast_ok(sh, Gate::LoPA)) {
    const int C = sh.d / W::EPC;
    const int cpl = cpl_for(C), lpr = lanes_per_row(C, cpl), lg = ilog2(lpr);
    const int rows_per_block = (kBlock / kWave) * 2 * (kWave >> lg);
    const int grid = (sh.r + rows_per_block - 1) / rows_per_block;
    if (cpl == 8)
      k_lopa_z_t1<W, 8><<<grid, kBlock, 0, s>>>(x, static_cast<const uint4*>(A), C, lpr, lg, sh.r, ws.z);
    else
      k_lopa_z_t1<W, 16><<<grid, kBlock, 0, s>>>(x, static_cast<const uint4*>(A), C, lpr, lg, sh.r, ws.z);
  } else {
    const int grid = (sh.r + kBlock / kWave - 1) / (kBlock / kWave);
    k_lopa_z_generic<W><<<grid, kBlock, 0, s>>>(x, A, sh.T, sh.d, sh.r, ws.z);
  }
  return hipGetLastError();
}

template <class W, bool DENSE>
hipError_t down(const Shape& sh, const void* w_down_t, const Workspace& ws, float* y, hipStream_t s) {
  const size_t shmem = DENSE ? 0 : sizeof(int) * (size_t)(ws.nseg + 1);
  if (sh.T == 1 && sh.d % W::EPC == 0) {
    constexpr int CPW = 16 / W::EPC;  // 16 output columns per workgroup
    const int C = sh.d / W::EPC;
    const int grid = (C + CPW - 1) / CPW;
    k_down_t1<W, CPW, DENSE><<<grid, kBlock, shmem, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff,
                                                        static_cast<const uint4*>(w_down_t), C, sh.d, y);
  } else {
    const int grid = (sh.d + kBlock - 1) / kBlock;
    k_down_generic<W, DENSE><<<grid, kBlock, shmem, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff,
                                                        ws.slots, w_down_t, sh.T, sh.d, y);
  }
  return hipGetLastError();
}

}  // namespace

// ------------------------------------------------------------------ launchers
hipError_t launch_lopa_z(const Shape& sh, const float* x, const void* lopa_a, const Workspace& ws, hipStream_t s) {
  return sh.wdt == 1 ? lopa_z<WBf16>(sh, x, lopa_a, ws, s) : lopa_z<WF32>(sh, x, lopa_a, ws, s);
}

hipError_t launch_gate_up(const Shape& sh, Gate g, bool dense, const float* x, const void* gate_w, const void* w_up,
                          float t, const Workspace& ws, hipStream_t s) {
  const bool lopa = g == Gate::LoPA;
  const bool fast = fast_ok(sh, g);
#define FFN_GU(W, L, D)                                                                     \
  return fast ? gate_up_fast<W, L, D>(sh, x, gate_w, w_up, t, ws, s)                       \
              : gate_up_generic<W, L, D>(sh, x, gate_w, w_up, t, ws, s)
  if (sh.wdt == 1) {
    if (lopa) {
      if (dense) FFN_GU(WBf16, true, true);
      FFN_GU(WBf16, true, false);
    }
    if (dense) FFN_GU(WBf16, false, true);
    FFN_GU(WBf16, false, false);
  }
  if (lopa) {
    if (dense) FFN_GU(WF32, true, true);
    FFN_GU(WF32, true, false);
  }
  if (dense) FFN_GU(WF32, false, true);
  FFN_GU(WF32, false, false);
#undef FFN_GU
}

hipError_t launch_down(const Shape& sh, bool dense, const void* w_down_t, const Workspace& ws, float* y,
                       hipStream_t s) {
  if (sh.wdt == 1) return dense ? down<WBf16, true>(sh, w_down_t, ws, y, s) : down<WBf16, false>(sh, w_down_t, ws, y, s);
  return dense ? down<WF32, true>(sh, w_down_t, ws, y, s) : down<WF32, false>(sh, w_down_t, ws, y, s);
}

}  // namespace ffn

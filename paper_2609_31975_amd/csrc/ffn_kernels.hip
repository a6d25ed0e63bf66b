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

// load_vec through raw buffer loads (zeros past C chunks): branch-free, and kept where it
// stands among the weight loads around it.
template <class W, int CPL>
__device__ __forceinline__ void load_vec_buf(const float* __restrict__ v, int C, int q, int lpr,
                                             float (&r)[CPL][W::EPC]) {
  constexpr int F4 = W::EPC / 4;  // float4s a chunk
  const Buf vb = make_buf(v, 16u * F4 * (uint32_t)C);
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = q + c * lpr;
#pragma unroll
    for (int e4 = 0; e4 < F4; ++e4) {
      const float4 f = __builtin_bit_cast(float4, ldb(vb, ch < C ? 16u * (uint32_t)(ch * F4 + e4) : kOOB));
      r[c][4 * e4 + 0] = f.x;
      r[c][4 * e4 + 1] = f.y;
      r[c][4 * e4 + 2] = f.z;
      r[c][4 * e4 + 3] = f.w;
    }
  }
}

// The vector a lane multiplies its chunks of a row with.  fp32 / bf16 weights: the fp32
// elements.  Quantized weights: X = rint(v * 127 * 2^16 / max |v|), a 24-bit fixed-point
// copy, kept as its three bytes: the signed top byte s2 and the unsigned bytes u1, u0,
// four elements a word, in the order the codes' words take them (int4: each code word
// gives a word of its even and one of its odd elements).  The dot products then run on
// v_dot4_i32_i8 (codes x s2) and v_dot4_u32_u8 (codes + 128, or int4 codes + 8, x u1 and
// x u0), and the per-lane sums of the limbs correct the offsets exactly in 32-bit
// integers; `scale` turns the sums back into the vector's units.  The workgroup converts
// the vector once, each thread a share, into LDS (prepare_lane_vec, called by dot_rows
// after its first weight loads); each lane then reads the words of its chunks.  The
// thread's share is loaded by make_lane_vec, ahead of the weights: loaded after them, its
// first use waited for the weights too (the load counter is in order).
// Q = false with quantized weights keeps the vector in fp32 and converts each code to
// fp32 (one op an int8 element, two an int4 one): twice the ALU work of the limbs or more,
// but no workgroup-wide conversion in front of the first row.  The kernels whose lanes
// multiply one row each (LoPA's z = A x and the W_up dots after LoPA's gate) take it;
// the gate streams, several rows a lane, keep the limbs (measured: fp32 z in LoPA's gate
// stream cost 1.3 us at int8 and 5 us at int4 on the 8B shape).
template <class W, int CPL, bool Q = is_quant<W>()>
struct LaneVec {
  float f[CPL][W::EPC];
};
// the representation of a vector multiplied with one row a lane: fp32 while a lane holds at
// most 64 elements
template <class W, int CPL>
constexpr bool limb_vec() {
  return is_quant<W>() && CPL * W::EPC > 64;
}
template <class W, int CPL>
struct LaneVec<W, CPL, true> {
  // int8: three byte limbs of X, four elements a word (limb 0 the signed top byte); int4: six
  // nibble limbs, eight elements a word, nibble k of a word holding element k as the codes do
  // (limb 0 the signed top nibble).  Either way four words a limb for a 16-byte chunk of codes.
  static constexpr int NL = W::LB == 8 ? 3 : 6;                   // limbs
  static constexpr int G = W::LB == 8 ? 4 : 8;                    // elements a thread converts at a time
  static constexpr int GPT = 8192 / G / kBlock;                   // groups a thread converts (up to 8192 elements)
  uint32_t limb[NL][CPL][4];
  int32_t lsum[NL];  // sums of each limb's values over the lane's elements
  float scale;
  float4 raw[GPT][G / 4];  // the thread's groups of the vector, until converted
  int C, q, lpr;
  bool ready;
};

template <class W, int CPL, bool Q>
__device__ __forceinline__ void make_lane_vec(const float* __restrict__ v, int C, int q, int lpr,
                                              LaneVec<W, CPL, Q>& out) {
  if constexpr (!Q) {
    load_vec<W, CPL>(v, C, q, lpr, out.f);
  } else {
    using LV = LaneVec<W, CPL, Q>;
    constexpr int G = LV::G;
    const int len = C * W::EPC, ngroups = len / G;
    const Buf vb = make_buf(v, 4u * (uint32_t)len);
#pragma unroll
    for (int i = 0; i < LV::GPT; ++i) {  // group g = threadIdx.x + i kBlock
      const int g = (int)threadIdx.x + i * kBlock;
#pragma unroll
      for (int h = 0; h < G / 4; ++h)
        out.raw[i][h] = __builtin_bit_cast(float4, ldb(vb, g < ngroups ? 16u * (uint32_t)(g * (G / 4) + h) : kOOB));
    }
    out.C = C;
    out.q = q;
    out.lpr = lpr;
    out.ready = false;
  }
}

// The quantized vector's limb words: kLimbSpace words, limb l at l * (8192 / G) (vectors up
// to 8192 elements; 24 KB for either format).
constexpr int kLimbSpace = 6144;

// Called by every thread of the workgroup at the same point (it has barriers).
template <class W, int CPL, bool Q>
__device__ __forceinline__ void prepare_lane_vec(LaneVec<W, CPL, Q>& out) {
  if constexpr (Q) {
    if (out.ready) return;
    out.ready = true;
    __shared__ uint32_t s_limb[kLimbSpace];
    __shared__ float s_max[2][kBlock / kWave];
    constexpr float kFull = 127.f * 65536.f;
    using LV = LaneVec<W, CPL, Q>;
    constexpr int G = LV::G, GPT = LV::GPT, NL = LV::NL, LW = 8192 / G;  // LW: words a limb
    const int len = out.C * W::EPC, ngroups = len / G;
    // the thread's groups: g = threadIdx.x + i * kBlock (zeros past the vector)
    const auto& vals = out.raw;
    float m = 0.f, nan = 0.f;
#pragma unroll
    for (int i = 0; i < GPT; ++i) {
#pragma unroll
      for (int h = 0; h < G / 4; ++h) {
        const float4 f = vals[i][h];
        m = fmaxf(fmaxf(fmaxf(m, fabsf(f.x)), fmaxf(fabsf(f.y), fabsf(f.z))), fabsf(f.w));
        nan += ((f.x * 0.f + f.y * 0.f) + (f.z * 0.f + f.w * 0.f));  // NaN if any is NaN or infinite
      }
    }
    m = wave_max(m);
    const float bad = wave_max(nan == 0.f ? 0.f : 1.f);
    const int wave = threadIdx.x / kWave;
    if (lane_id() == 0) {
      s_max[0][wave] = m;
      s_max[1][wave] = bad;
    }
    __syncthreads();
    float mm = 0.f, bb = 0.f;
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w) {
      mm = fmaxf(mm, s_max[0][w]);
      bb = fmaxf(bb, s_max[1][w]);
    }
    const float k = (bb == 0.f && mm > 0.f) ? kFull / mm : 0.f;
    out.scale = bb != 0.f ? __builtin_nanf("") : mm / kFull;
#pragma unroll
    for (int i = 0; i < GPT; ++i) {
      const int g = (int)threadIdx.x + i * kBlock;
      if (g < ngroups) {
        int X[G];
#pragma unroll
        for (int h = 0; h < G / 4; ++h) {  // |e k| <= kFull (NaN: clamped, the scale is NaN then)
          const float e[4] = {vals[i][h].x, vals[i][h].y, vals[i][h].z, vals[i][h].w};
#pragma unroll
          for (int b = 0; b < 4; ++b) X[4 * h + b] = (int)rintf(fminf(fmaxf(e[b] * k, -kFull), kFull));
        }
        if constexpr (W::LB == 8) {
          // byte j of X0..X3 into one word per j (v_perm_b32: selector bytes 0-3 pick the
          // second operand's bytes, 4-7 the first's, 12 gives zero)
          const uint32_t lo = __builtin_amdgcn_perm((uint32_t)X[1], (uint32_t)X[0], 0x06020400u);  // X0.b0 X1.b0 X0.b2 X1.b2
          const uint32_t hi = __builtin_amdgcn_perm((uint32_t)X[3], (uint32_t)X[2], 0x06020400u);  // X2.b0 X3.b0 X2.b2 X3.b2
          const uint32_t mid = __builtin_amdgcn_perm((uint32_t)X[1], (uint32_t)X[0], 0x0c0c0501u);  // X0.b1 X1.b1 0 0
          const uint32_t mid2 = __builtin_amdgcn_perm((uint32_t)X[3], (uint32_t)X[2], 0x0c0c0501u); // X2.b1 X3.b1 0 0
          s_limb[0 * LW + g] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);     // byte 2 of X0..X3
          s_limb[1 * LW + g] = __builtin_amdgcn_perm(mid2, mid, 0x05040100u);  // byte 1
          s_limb[2 * LW + g] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);     // byte 0
        } else {
          // nibble 5 - l of X0..X7 into word l, nibble k of the word from X_k (X fits 24 bits
          // signed, so its top nibble is the signed limb)
#pragma unroll
          for (int l = 0; l < 6; ++l) {
            uint32_t wd = 0u;
#pragma unroll
            for (int b = 0; b < 8; ++b) wd |= (((uint32_t)X[b] >> (4 * (5 - l))) & 15u) << (4 * b);
            s_limb[l * LW + g] = wd;
          }
        }
      }
    }
    __syncthreads();
    int32_t ls[NL];
#pragma unroll
    for (int l = 0; l < NL; ++l) ls[l] = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int ch = out.q + c * out.lpr;
#pragma unroll
      for (int wi = 0; wi < 4; ++wi) {
        const bool ok = ch < out.C;
        const int word = ch * 4 + wi;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          const uint32_t wl = ok ? s_limb[l * LW + word] : 0u;
          out.limb[l][c][wi] = wl;
          if constexpr (W::LB == 8)
            ls[l] = l == 0 ? __builtin_amdgcn_sdot4((int)wl, 0x01010101, ls[l], false)
                           : (int32_t)__builtin_amdgcn_udot4(wl, 0x01010101u, (uint32_t)ls[l], false);
          else
            ls[l] = l == 0 ? __builtin_amdgcn_sdot8((int)wl, 0x11111111, ls[l], false)
                           : (int32_t)__builtin_amdgcn_udot8(wl, 0x11111111u, (uint32_t)ls[l], false);
        }
      }
    }
#pragma unroll
    for (int l = 0; l < NL; ++l) out.lsum[l] = ls[l];
    __syncthreads();  // the limb words are read before any later conversion overwrites them
  }
}

template <class W, int CPL, bool Q>
__device__ __forceinline__ float lane_dot(const uint4 (&b)[CPL], const LaneVec<W, CPL, Q>& v) {
  if constexpr (!Q) {
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float f[W::EPC];
      unpack(W{}, b[c], f);
#pragma unroll
      for (int e = 0; e < W::EPC; e += 2) {
        acc0 = fmaf(f[e], v.f[c][e], acc0);
        acc1 = fmaf(f[e + 1], v.f[c][e + 1], acc1);
      }
    }
    return acc0 + acc1;
  } else if constexpr (W::LB == 8) {
    int32_t a2 = 0;
    uint32_t a1 = 0u, a0 = 0u;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const uint32_t cw[4] = {b[c].x, b[c].y, b[c].z, b[c].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {  // signed codes w; w ^ 0x80 per byte = w + 128
        const uint32_t off = cw[i] ^ 0x80808080u;
        a2 = __builtin_amdgcn_sdot4((int)cw[i], (int)v.limb[0][c][i], a2, false);
        a1 = __builtin_amdgcn_udot4(off, v.limb[1][c][i], a1, false);
        a0 = __builtin_amdgcn_udot4(off, v.limb[2][c][i], a0, false);
      }
    }
    // remove the code offsets: sum (w + 128) u = sum w u + 128 sum u
    const int32_t e2 = a2;
    const int32_t e1 = (int32_t)a1 - 128 * v.lsum[1], e0 = (int32_t)a0 - 128 * v.lsum[2];
    return fmaf((float)e2, 65536.f, fmaf((float)e1, 256.f, (float)e0)) * v.scale;
  } else {
    // int4: v_dot8 of eight nibbles at a time; the signed top limb against the signed codes,
    // the five unsigned limbs against the codes + 8 (nibble ^ 8)
    int32_t a5 = 0;
    uint32_t au[5] = {0u, 0u, 0u, 0u, 0u};
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const uint32_t cw[4] = {b[c].x, b[c].y, b[c].z, b[c].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t off = cw[i] ^ 0x88888888u;
        a5 = __builtin_amdgcn_sdot8((int)cw[i], (int)v.limb[0][c][i], a5, false);
#pragma unroll
        for (int l = 1; l < 6; ++l) au[l - 1] = __builtin_amdgcn_udot8(off, v.limb[l][c][i], au[l - 1], false);
      }
    }
    float r = 0.f;
#pragma unroll
    for (int l = 5; l >= 1; --l) {  // nibble 0 (l = 5) up to nibble 4 (l = 1), then the top one
      const int32_t e = (int32_t)au[l - 1] - 8 * v.lsum[l];
      r = fmaf((float)e, (float)(1 << (4 * (5 - l))), r);
    }
    return fmaf((float)a5, 1048576.f, r) * v.scale;
  }
}

// The sum over the 64 lanes, the same in every lane: the rows of 16 lanes reduce by DPP and
// their four sums are read with v_readlane, with no LDS round trip (group_sum's last two
// steps are lane shuffles through LDS).  The same additions in the same order as
// group_sum(v, 64), so the result is bit-identical.  Every lane must be active.
__device__ __forceinline__ float wave_sum_uniform(float r) {
  r += dpp_move<kDppXor1>(r);
  r += dpp_move<kDppXor2>(r);
  r += dpp_move<kDppHalfMirror>(r);
  r += dpp_move<kDppMirror>(r);
  const int ri = __float_as_int(r);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(ri, 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(ri, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(ri, 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(ri, 48));
  return (r0 + r1) + (r2 + r3);
}

// Dot products <rows, v> for rows picked by `row_of(k)`, k in [0, n), of a matrix of
// `bytes` bytes (< 2^31): each wave takes passes of 64/lpr rows (passes wave, wave + 4,
// ...).  For rows of at most 8 chunks per lane and more than one pass per wave, two
// register sets alternate, the loads of the next pass issued before the current pass is
// reduced (measured: preloading both sets, or four sets, around the quantized vector's
// conversion ran slower); the loads are raw buffer loads
// (out-of-range offsets past the last pass), so every pass issues the same loads and the
// load-counter waits are exact.  A group of passes always runs whole (a pass past the
// last one loads nothing and sinks nothing) and the exit test closes the group, so no
// load sits on a conditional path.
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

// LATE = 2: the same, from the float4s of an LDS copy `lds_vec` (zeros past C chunks).
// LATE (fp32 vectors only): v is loaded here from `vec`, after the first pass's row loads,
// so that the weight stream starts ahead of the vector loads of all the waves on a CU.  It
// pays for long streams (the standard gate); for a stream of one pass (LoPA's z and gate,
// the W_up dots after LoPA's gate) the in-order load counter makes the first use of the
// vector wait for all the rows, and the call measured slower.
// `stage` runs right after the first pass's row loads, in every thread of the workgroup
// (LATE = 2: it may fill lds_vec, and ends with a barrier then).
struct NoStage {
  __device__ void operator()() const {}
};
// `pre` runs before the first pass's row loads (loads it issues are ahead of them in the
// in-order load counter, so that `stage` can wait for them without waiting for the rows).
template <class W, int CPL, int LATE = 0, bool Q, class RowOf, class Sink, class Stage = NoStage, class Pre = NoStage>
__device__ __forceinline__ void dot_rows(const uint4* __restrict__ mat, uint32_t bytes, int C, int lpr, int lpr_log2,
                                         int n, LaneVec<W, CPL, Q>& v, RowOf row_of, Sink sink,
                                         const float* __restrict__ vec = nullptr, const float4* lds_vec = nullptr,
                                         Stage stage = Stage{}, Pre pre = Pre{}) {
  static_assert(!(LATE && Q), "a late vector is an fp32 one");
  constexpr int kWaves = kBlock / kWave;
  const Buf mb = make_buf(mat, bytes);
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const int q = lane & (lpr - 1), p = lane >> lpr_log2;
  const int rpp = kWave >> lpr_log2;
  const int npass = (n + rpp - 1) / rpp;
  auto load = [&](uint4 (&b)[CPL], int pass) {
    const int k = pass * rpp + p;
    const bool ok = pass < npass && k < n;
    load_pass<W, CPL>(mb, C, q, lpr, ok, ok ? row_of(k) : 0, b);
  };
  auto finish = [&](const uint4 (&b)[CPL], int pass) {
    const int k = pass * rpp + p;
    const float dot = lane_dot<W, CPL, Q>(b, v);
    const float sum = lpr == kWave ? wave_sum_uniform(dot) : group_sum(dot, lpr);
    if (q == 0 && k < n) sink(k, sum);
  };
  uint4 b0[CPL], b1[CPL];
  constexpr bool kPre = !__is_same(Pre, NoStage);
  if constexpr (kPre) {
    pre();
    issue_barrier();
  }
  load(b0, wave);  // a wave without passes loads nothing (out-of-range offsets)
  if constexpr (kPre) issue_barrier();
  stage();
  if constexpr (LATE == 1) {
    issue_barrier();
    load_vec_buf<W, CPL>(vec, C, q, lpr, v.f);
    issue_barrier();
  } else if constexpr (LATE == 2) {
    constexpr int F4 = W::EPC / 4;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
#pragma unroll
      for (int e4 = 0; e4 < F4; ++e4) {
        const float4 f = lds_vec[(q + c * lpr) * F4 + e4];
        v.f[c][4 * e4 + 0] = f.x;
        v.f[c][4 * e4 + 1] = f.y;
        v.f[c][4 * e4 + 2] = f.z;
        v.f[c][4 * e4 + 3] = f.w;
      }
    }
  }
  prepare_lane_vec<W, CPL, Q>(v);  // limbs: the whole workgroup converts the vector
  if (wave >= npass) return;
  if (wave + kWaves >= npass) {  // a single pass: nothing to overlap
    finish(b0, wave);
    return;
  }
  if constexpr (CPL <= 8) {
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

// Standard gating with one row per wave a pass (64 lanes a row): the gate rows and the W_up
// rows of the active neurons go through one stream.  A step finishes the row in one buffer
// and reloads that buffer: with the W_up row of the same neuron when its gate value exceeds
// t, else with the wave's next gate row.  The W_up reads of a segment thus overlap its gate
// stream instead of following its compaction, and only an active last gate row costs a
// round trip after the stream.  Every step issues the same loads (a buffer with nothing left
// to load gets out-of-range offsets), so the load-counter waits stay exact; what a step does
// next is uniform over the wave (all lanes hold the same group sum).  Gate values go to
// s_h[k]; an active row's zval (activation value times the W_up dot, SiLU'd with
// form.silu_up) goes to s_zv[k].  gate_w and w_up are both [d_ff][C] chunks of `bytes`.
// The wave's first gate row is requested before x and its second after it, so that the weight
// stream starts ahead of the vector loads of all the waves on a CU.
template <class W, int CPL, bool FULL>
__device__ __forceinline__ void gate_up_stream(const float* __restrict__ x, const uint4* __restrict__ gate_w,
                                               const uint4* __restrict__ w_up, uint32_t bytes, int C, int row0, int n,
                                               float t, const Form& form, float* s_h, float* s_zv) {
  constexpr int kWaves = kBlock / kWave;
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const int act = FULL ? form.act : 0;
  int next_gate = wave;
  LaneVec<W, CPL, false> v;
  // a buffer's work: kind 1 the gate row k, kind 2 the W_up row k with activation value a,
  // kind 0 nothing
  struct Item {
    int kind, k;
    float a;
  };
  auto take_gate = [&](Item& it) {
    it.kind = next_gate < n ? 1 : 0;
    it.k = next_gate;
    next_gate += kWaves;
  };
  auto load = [&](uint4 (&b)[CPL], const Item& it) {
    const Buf mb = make_buf(it.kind == 2 ? w_up : gate_w, bytes);
    load_pass<W, CPL>(mb, C, lane, kWave, it.kind != 0, row0 + it.k, b);
  };
  auto finish = [&](const uint4 (&b)[CPL], Item& it) {
    if (it.kind == 0) return;
    const float s = wave_sum_uniform(lane_dot<W, CPL, false>(b, v));
    if (it.kind == 1) {
      if (lane == 0) s_h[it.k] = s;
      if (s > t) {  // NaN compares false: inactive
        it.kind = 2;
        it.a = gate_value(act, s - t);
        return;
      }
    } else if (lane == 0) {
      s_zv[it.k] = it.a * (FULL ? up_value(form.silu_up, s) : s);
    }
    take_gate(it);
  };
  uint4 b0[CPL];
  Item i0, i1;
  take_gate(i0);
  load(b0, i0);
  issue_barrier();
  // x is loaded once per workgroup (each thread a share, zeros past its C chunks) and staged
  // in LDS, from where every lane reads its chunks
  constexpr int F4 = W::EPC / 4, kXF4 = CPL * kWave * F4, kXPT = kXF4 / kBlock;
  static_assert(kXPT * kBlock == kXF4, "x shares");
  __shared__ float4 s_x[kXF4];
  float4 xs[kXPT];
  {
    const int nf4 = C * F4;
    const Buf xb = make_buf(x, 16u * (uint32_t)nf4);
#pragma unroll
    for (int k = 0; k < kXPT; ++k) {
      const int j = (int)threadIdx.x + k * kBlock;
      xs[k] = __builtin_bit_cast(float4, ldb(xb, j < nf4 ? 16u * (uint32_t)j : kOOB));
    }
  }
  issue_barrier();
  auto stage_x = [&] {
#pragma unroll
    for (int k = 0; k < kXPT; ++k) s_x[threadIdx.x + k * kBlock] = xs[k];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
#pragma unroll
      for (int e4 = 0; e4 < F4; ++e4) {
        const float4 f = s_x[(lane + c * kWave) * F4 + e4];
        v.f[c][4 * e4 + 0] = f.x;
        v.f[c][4 * e4 + 1] = f.y;
        v.f[c][4 * e4 + 2] = f.z;
        v.f[c][4 * e4 + 3] = f.w;
      }
    }
  };
  if constexpr (CPL <= 8) {
    uint4 b1[CPL];
    take_gate(i1);
    load(b1, i1);
    issue_barrier();
    stage_x();
    while (true) {
      finish(b0, i0);
      load(b0, i0);
      issue_barrier();
      finish(b1, i1);
      load(b1, i1);
      issue_barrier();
      if (i0.kind == 0 && i1.kind == 0) break;
    }
  } else {
    stage_x();
    while (true) {
      finish(b0, i0);
      if (i0.kind == 0) break;
      load(b0, i0);
      issue_barrier();
    }
  }
}

// Ballot compaction of one segment (run by the first wave): neurons whose gate value
// exceeds t (all neurons if `all`) get ascending ranks; their activation value (h - t,
// or its R-S+ with act = 1) is kept in LDS for the W_up phase and published with the
// neuron index.
// With s_zv, the zval of each selected neuron is already in s_zv[row] and is published too.
__device__ __forceinline__ void compact_segment(const float* s_h, int nrows, int row0, int seg, float t, bool all,
                                                int act, int* s_list, float* s_act, int* s_cnt, int32_t* seg_count,
                                                int32_t* seg_idx, float* seg_act, const float* s_zv = nullptr,
                                                float* seg_zval = nullptr) {
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
      if (s_zv) seg_zval[row0 + rank] = s_zv[lane];
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
                                                      GWork gw, const float* __restrict__ s_a) {
  if (g_precompute(gw)) return;
  __shared__ float s_z[kBlock];  // quantized: the block's sums before their row scales
  LaneVec<W, CPL, limb_vec<W, CPL>()> xr;
  make_lane_vec<W, CPL>(x, C, lane_id() & (lpr - 1), lpr, xr);
  const int rows_per_block = (kBlock / kWave) * (kWave >> lpr_log2);
  const int k0 = blockIdx.x * rows_per_block;
  const int n = min(rows_per_block, r - k0);
  auto put = [&](int k, float s) {
    if constexpr (NORM) {
      z[k0 + k] = gain ? s * gain[k0 + k] : s;
      zsq[k0 + k] = s * s;
    } else {
      z[k0 + k] = s;
    }
  };
  // quantized: thread i's row scale, loaded before the stream and applied after it
  const float sa = is_quant<W>() ? __builtin_bit_cast(float, ldb32(make_buf(s_a, 4u * (uint32_t)r),
                                                                   (int)threadIdx.x < n
                                                                       ? 4u * (uint32_t)(k0 + (int)threadIdx.x)
                                                                       : kOOB))
                                 : 1.f;
  dot_rows<W, CPL>(A, 16u * (uint32_t)r * (uint32_t)C, C, lpr, lpr_log2, n, xr, [&](int k) { return k0 + k; },
                   [&](int k, float s) {
                     if constexpr (is_quant<W>())
                       s_z[k] = s;
                     else
                       put(k, s);
                   });
  if constexpr (is_quant<W>()) {
    __syncthreads();
    if ((int)threadIdx.x < n) put(threadIdx.x, s_z[threadIdx.x] * sa);
  }
}

// z = A x for one token with fp32 / bf16 rows, one row a workgroup: thread i takes chunks
// i, i + 256, ... (CPL of them) of the row and of x, and the wave sums meet in LDS.  Each
// thread keeps a handful of loads in flight, and the rows spread over every CU (the
// one-row-a-wave kernel above gives 4 rows a workgroup and half the CUs at r = 512).
template <class W, int CPL, bool NORM>
__global__ __launch_bounds__(kBlock) void k_lopa_z_row(const float* __restrict__ x, const uint4* __restrict__ A,
                                                       int C, int r, float* __restrict__ z,
                                                       const float* __restrict__ gain, float* __restrict__ zsq,
                                                       GWork gw) {
  if (g_precompute(gw)) return;
  __shared__ float s_p[kBlock / kWave];
  const int k = blockIdx.x;
  LaneVec<W, CPL, false> v;
  load_vec_buf<W, CPL>(x, C, threadIdx.x, kBlock, v.f);
  const Buf ab = make_buf(A, 16u * (uint32_t)r * (uint32_t)C);
  uint4 b[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = (int)threadIdx.x + c * kBlock;
    b[c] = ldb_nt(ab, ch < C ? 16u * ((uint32_t)k * (uint32_t)C + (uint32_t)ch) : kOOB);
  }
  const float part = wave_sum_uniform(lane_dot<W, CPL, false>(b, v));
  if (lane_id() == 0) s_p[threadIdx.x / kWave] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w) sum += s_p[w];
    if constexpr (NORM) {
      z[k] = gain ? sum * gain[k] : sum;
      zsq[k] = sum * sum;
    } else {
      z[k] = sum;
    }
  }
}

// One segment: gate values, compaction, W_up dots of the selected neurons.
// LOPA: the gate rows are B [d_ff][r] against z; otherwise W_gate [d_ff][d] against x.
// DENSE: every neuron of the segment is selected (act = max(h - t, 0)).
// FORM (a FormKind): the paper's full form (`form`): the activation value, SiLU on the
// W_up output and, with kFormLoPA, the fixed term G and RMSNorm of z.
// CPLA > 0 (LoPA, fp32 / bf16 rows): z = A x is computed inside this kernel instead of by a
// kernel before it.  Workgroup w computes the z components of range w of Split(r, nseg) (the
// first r workgroups one each when r <= nseg), CPLA chunks of an A row (and of x) a thread,
// and publishes each with one 64-bit store, the value and kZTag together; it then reads all
// r components back, each with one 64-bit load, until every tag is there.  The loads of the
// A rows go out first, then the workgroup's B rows, so that the rows stream while z is formed
// and handed over, and the wait for z covers only the A rows.  The down kernel of the call
// clears the tags.  A workgroup that has not seen every component after form.z_wait ticks
// (kZWaitTicks unless a test shortens it) computes the missing ones itself, so the kernel
// finishes whatever the residency of its workgroups.
template <class W, bool LOPA, bool DENSE, int CPLG, int CPLU, int FORM, int CPLA = 0>
__global__ __launch_bounds__(kBlock) void k_gate_up_t1(const float* __restrict__ x, const float* __restrict__ z,
                                                       const uint4* __restrict__ gate_w, int Cg, int lprg,
                                                       int lprg_log2, const uint4* __restrict__ w_up, int Cu,
                                                       int lpru, int lpru_log2, int d_ff, int nseg, float t,
                                                       int32_t* __restrict__ meta, int32_t* __restrict__ seg_count,
                                                       int32_t* __restrict__ seg_idx, float* __restrict__ seg_act,
                                                       float* __restrict__ seg_zval, float* __restrict__ y, int d,
                                                       Form form, const float* __restrict__ zsq,
                                                       const float* __restrict__ gx, const float* __restrict__ s_g,
                                                       const float* __restrict__ s_up, const uint4* __restrict__ A,
                                                       uint64_t* __restrict__ zslot) {
  constexpr bool FULL = FORM != kFormDefault, EXTRA = LOPA && FORM == kFormLoPA;
  constexpr bool FZ = LOPA && CPLA > 0;
  static_assert(!FZ || (!is_quant<W>() && CPLG <= 8), "z is computed in the gate kernel for fp32 / bf16 rows");
  __shared__ float s_h[kSegMax];
  __shared__ float s_ss[kBlock / kWave];
  __shared__ int s_list[kSegMax];
  __shared__ float s_act[kSegMax];
  __shared__ float s_usc[kSegMax];  // quantized: the W_up row scales of the segment
  __shared__ int s_cnt;

  const int seg = blockIdx.x;
  const Split segs(d_ff, nseg);
  const int row0 = segs.start(seg);
  const int nrows = segs.start(seg + 1) - row0;
  clear_output(y, d, meta, nseg);
  // quantized: thread i's row scales (gate, W_up), loaded branch-free before the streams and
  // applied after the gate stream, so that no load waits inside a stream
  const bool own = (int)threadIdx.x < nrows;
  const uint32_t srow = own ? 4u * (uint32_t)(row0 + (int)threadIdx.x) : kOOB;
  const float sg = is_quant<W>() ? __builtin_bit_cast(float, ldb32(make_buf(s_g, 4u * (uint32_t)d_ff), srow)) : 1.f;
  const float su = is_quant<W>() ? __builtin_bit_cast(float, ldb32(make_buf(s_up, 4u * (uint32_t)d_ff), srow)) : 1.f;
  auto gate_sink = [&](int k, float s) { s_h[k] = s; };
  auto gate_row = [&](int k) { return row0 + k; };
  auto up_row = [&](int e) { return row0 + s_list[e]; };
  auto up_sink = [&](int e, float v) {
    if constexpr (is_quant<W>()) v *= s_usc[s_list[e]];
    seg_zval[row0 + e] = s_act[e] * (FULL ? up_value(form.silu_up, v) : v);
  };
  // after the gate stream: the gate's row scales, and the W_up ones to LDS
  auto apply_scales = [&] {
    if constexpr (is_quant<W>()) {
      if (own) {
        s_h[threadIdx.x] *= sg;
        s_usc[threadIdx.x] = su;
      }
      __syncthreads();
    }
  };
  const int act = FULL ? form.act : 0;

  if constexpr (LOPA) {
    // x for the W_up dots (fp32 vectors, one row a wave): loaded once per workgroup, each
    // thread a share, ahead of the gate stream, and staged in LDS during the compaction, so
    // that the W_up rows go out right after it (every wave reading 16 KB of x there had put
    // 50 MB of L2 reads in front of the 12 MB of W_up rows)
    constexpr bool kXLds = !limb_vec<W, CPLU>() && CPLU <= 8 && !DENSE;
    constexpr int XF4 = W::EPC / 4, kXF4 = kXLds ? CPLU * kWave * XF4 : kBlock, kXPT = kXF4 / kBlock;
    static_assert(kXPT * kBlock == kXF4, "x shares");
    __shared__ float4 s_xu[kXLds ? kXF4 : 1];
    const bool xlds = kXLds && lpru == kWave;
    float4 xs[kXPT];
    if constexpr (kXLds) {
      const int nf4 = Cu * XF4;
      const Buf xb = make_buf(x, 16u * (uint32_t)nf4);
#pragma unroll
      for (int k = 0; k < kXPT; ++k) {
        const int j = (int)threadIdx.x + k * kBlock;
        xs[k] = __builtin_bit_cast(float4, ldb(xb, xlds && j < nf4 ? 16u * (uint32_t)j : kOOB));
      }
    }
    // LoPA's fixed term (G x)_i of this thread's row (written by the z kernel's extra
    // workgroups, or gathered here when z is computed here) and the squares of z for RMSNorm:
    // loaded before the gate stream, used after it, branch-free so that nothing waits for
    // them in front of the stream
    const bool has_g = EXTRA && form.g_idx;
    const bool own_row = (int)threadIdx.x < nrows;
    uint32_t gbits = 0u;
    GEntry gent{0u, 0.f};
    if constexpr (EXTRA && !FZ)
      gbits = ldb32(make_buf(gx, 4u * (uint32_t)d_ff), has_g && own_row ? 4u * (uint32_t)(row0 + (int)threadIdx.x)
                                                                        : kOOB);
    if constexpr (EXTRA && FZ) gent = g_fetch(form, d_ff, has_g && own_row ? row0 + (int)threadIdx.x : -1);
    const bool norm = EXTRA && form.rms_eps > 0.f;
    const int r = Cg * W::EPC;
    uint32_t sq[EXTRA && !FZ ? kNormRegs : 1] = {};
    if constexpr (EXTRA && !FZ) {
      const Buf qb = make_buf(zsq, 4u * (uint32_t)r);
#pragma unroll
      for (int j = 0; j < kNormRegs; ++j) {
        const int k = (int)threadIdx.x + j * kBlock;
        sq[j] = ldb32(qb, norm && k < r ? 4u * (uint32_t)k : kOOB);
      }
    }
    float inv = 1.f;  // RMSNorm's 1 / sqrt(mean z^2 + eps) (fused z: found while z is staged)
    {
      LaneVec<W, CPLG> zr;  // limbs: the B stream gives a lane several rows
      // fp32 z: loaded once per workgroup (each thread a share) ahead of the B rows and
      // staged in LDS once the rows are requested, instead of 16 KB of z reads a wave
      constexpr bool kZLds = !is_quant<W>() && CPLG <= 8;
      if constexpr (kZLds) {
        constexpr int ZF4 = W::EPC / 4, kZF4 = CPLG * kWave * ZF4, kZPT = kZF4 / kBlock;
        static_assert(kZPT * kBlock == kZF4, "z shares");
        __shared__ float4 s_zs[kZF4];
        if constexpr (FZ) {
          // z = A x here (see above the kernel).  Components of this workgroup: [zk0, zk0 + nz)
          constexpr int ZR = 2, AF4 = W::EPC / 4, kZC = kFusedZMax / kBlock;
          const int Ca = d / W::EPC;
          const Split zsp(r, nseg);
          const int zk0 = zsp.start(seg), nz = zsp.start(seg + 1) - zk0;
          const Buf ab = make_buf(A, 16u * (uint32_t)r * (uint32_t)Ca);
          uint4 ar[ZR][CPLA];
          LaneVec<W, CPLA, false> xa;
          auto load_a = [&](int zb) {
#pragma unroll
            for (int zr_ = 0; zr_ < ZR; ++zr_)
#pragma unroll
              for (int c = 0; c < CPLA; ++c) {
                const int ch = (int)threadIdx.x + c * kBlock;
                ar[zr_][c] = ldb_nt(ab, zb + zr_ < nz && ch < Ca ? 16u * ((uint32_t)(zk0 + zb + zr_) * (uint32_t)Ca +
                                                                          (uint32_t)ch)
                                                                 : kOOB);
              }
          };
          __shared__ float s_zp[ZR][kBlock / kWave];
          float* const s_zf = reinterpret_cast<float*>(s_zs);
          // components zb .. zb + ZR - 1 of the workgroup, their A rows loaded: partial sums of the
          // thread's chunks, the 64 lanes, then the four waves in order, as the z kernel adds
          // them; each goes out with one 64-bit store, its tag in the high word
          auto publish = [&](int zb) {
            const int wave = threadIdx.x / kWave;
            float part[ZR];
#pragma unroll
            for (int zr_ = 0; zr_ < ZR; ++zr_) part[zr_] = wave_sum_uniform(lane_dot<W, CPLA, false>(ar[zr_], xa));
            if (lane_id() == 0)
#pragma unroll
              for (int zr_ = 0; zr_ < ZR; ++zr_) s_zp[zr_][wave] = part[zr_];
            __syncthreads();
            if ((int)threadIdx.x < min(ZR, nz - zb)) {
              const float s = ((s_zp[threadIdx.x][0] + s_zp[threadIdx.x][1]) + s_zp[threadIdx.x][2]) +
                              s_zp[threadIdx.x][3];
              const uint64_t word = ((uint64_t)kZTag << 32) | (uint64_t)__float_as_uint(s);
              __hip_atomic_store(zslot + zk0 + zb + threadIdx.x, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();
          };
          // A workgroup that computes components does so before it requests its B rows: its A
          // rows then share the memory system with the other workgroups' B rows only, and z is
          // out about a round trip after the kernel starts (measured: with the B rows requested
          // first, the last component went out 6.5 us into the kernel and z was complete
          // everywhere at 9 us)
          auto pre = [&] {
            load_a(0);
            const Buf xb = make_buf(x, 16u * AF4 * (uint32_t)Ca);
#pragma unroll
            for (int c = 0; c < CPLA; ++c) {
              const int ch = (int)threadIdx.x + c * kBlock;
#pragma unroll
              for (int e4 = 0; e4 < AF4; ++e4) {
                const float4 f = __builtin_bit_cast(
                    float4, ldb(xb, nz > 0 && ch < Ca ? 16u * (uint32_t)(ch * AF4 + e4) : kOOB));
                xa.f[c][4 * e4 + 0] = f.x;
                xa.f[c][4 * e4 + 1] = f.y;
                xa.f[c][4 * e4 + 2] = f.z;
                xa.f[c][4 * e4 + 3] = f.w;
              }
            }
            if (nz > 0) publish(0);  // workgroup-uniform
          };
          auto stage = [&] {
            const int wave = threadIdx.x / kWave;
            if constexpr (EXTRA) gbits = g_gather_bits(gent, x, d, has_g && own_row);
            // 1) components past the first ZR (r > ZR nseg): after the B rows
            for (int zb = ZR; zb < nz; zb += ZR) {  // workgroup-uniform
              load_a(zb);
              publish(zb);
            }
            // 2) every component, through its tag: thread i holds components i, i + 256, ...
            float zv[kZC];
            bool have[kZC];
#pragma unroll
            for (int i = 0; i < kZC; ++i) {
              zv[i] = 0.f;
              have[i] = (int)threadIdx.x + i * kBlock >= r;
            }
            const uint64_t t0 = wall_clock64();
            bool late = false;
            for (;;) {
              bool all = true;
#pragma unroll
              for (int i = 0; i < kZC; ++i) {
                if (!have[i]) {
                  const uint64_t v = __hip_atomic_load(zslot + threadIdx.x + i * kBlock, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                  if ((uint32_t)(v >> 32) == kZTag) {
                    have[i] = true;
                    zv[i] = __uint_as_float((uint32_t)v);
                  } else {
                    all = false;
                  }
                }
              }
              if (__syncthreads_and(all)) break;
              if (__syncthreads_or(wall_clock64() - t0 > form.z_wait)) {
                late = true;
                break;
              }
              __builtin_amdgcn_s_sleep(2);
            }
            // 3) into LDS (zeros past r, which the lanes' last chunks may read); a component
            // still missing is marked with the tag pattern and computed here, a wave a row
#pragma unroll
            for (int i = 0; i < kZF4 * 4 / kBlock; ++i) {
              const int j = (int)threadIdx.x + i * kBlock;
              s_zf[j] = i < kZC && j < r ? (have[i] ? zv[i] : __uint_as_float(kZTag)) : 0.f;
            }
            __syncthreads();
            if (late) {  // workgroup-uniform
              const Buf xb = make_buf(x, 16u * AF4 * (uint32_t)Ca);
              for (int k = wave; k < r; k += kBlock / kWave) {
                if (__float_as_uint(s_zf[k]) != kZTag) continue;  // wave-uniform (one LDS word)
                float s = 0.f;
                for (int ch = lane_id(); ch < Ca; ch += kWave) {
                  float f[W::EPC];
                  unpack(W{}, ldb(ab, 16u * ((uint32_t)k * (uint32_t)Ca + (uint32_t)ch)), f);
#pragma unroll
                  for (int e4 = 0; e4 < AF4; ++e4) {
                    const float4 xv = __builtin_bit_cast(float4, ldb(xb, 16u * (uint32_t)(ch * AF4 + e4)));
                    s = fmaf(f[4 * e4], xv.x, fmaf(f[4 * e4 + 1], xv.y, fmaf(f[4 * e4 + 2], xv.z,
                                                                              fmaf(f[4 * e4 + 3], xv.w, s))));
                  }
                }
                s = wave_sum(s);
                if (lane_id() == 0) s_zf[k] = s;
              }
              __syncthreads();
#pragma unroll
              for (int i = 0; i < kZC; ++i)
                if ((int)threadIdx.x + i * kBlock < r) zv[i] = s_zf[threadIdx.x + i * kBlock];
              __syncthreads();
            }
            // 4) RMSNorm: the scale from every component's square; z goes to LDS times the gains
            if constexpr (EXTRA) {
              if (norm) {  // workgroup-uniform
                float ss = 0.f;
#pragma unroll
                for (int i = 0; i < kZC; ++i) ss += zv[i] * zv[i];
                ss = wave_sum(ss);
                if (lane_id() == 0) s_ss[wave] = ss;
                __syncthreads();
                float tot = 0.f;
#pragma unroll
                for (int w = 0; w < kBlock / kWave; ++w) tot += s_ss[w];
                inv = 1.f / sqrtf(tot / (float)r + form.rms_eps);
                if (form.rms_gain) {
#pragma unroll
                  for (int i = 0; i < kZC; ++i) {
                    const int j = (int)threadIdx.x + i * kBlock;
                    if (j < r) s_zf[j] = zv[i] * form.rms_gain[j];
                  }
                }
                __syncthreads();
              }
            }
          };
          dot_rows<W, CPLG, 2>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, zr, gate_row,
                               gate_sink, nullptr, s_zs, stage, pre);
        } else {
          float4 zs[kZPT];
          const int nf4 = Cg * ZF4;
          const Buf zb = make_buf(z, 16u * (uint32_t)nf4);
#pragma unroll
          for (int k = 0; k < kZPT; ++k) {
            const int j = (int)threadIdx.x + k * kBlock;
            zs[k] = __builtin_bit_cast(float4, ldb(zb, j < nf4 ? 16u * (uint32_t)j : kOOB));
          }
          issue_barrier();
          auto stage = [&] {
#pragma unroll
            for (int k = 0; k < kZPT; ++k) s_zs[threadIdx.x + k * kBlock] = zs[k];
            __syncthreads();
          };
          dot_rows<W, CPLG, 2>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, zr,
                               gate_row, gate_sink, nullptr, s_zs, stage);
        }
      } else {
        make_lane_vec<W, CPLG>(z, Cg, lane_id() & (lprg - 1), lprg, zr);
        dot_rows<W, CPLG>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, zr, gate_row,
                          gate_sink);
      }
    }
    // G x: the z kernel's extra workgroups stored g_sign x[g_idx]; gathered here, the sign
    // is applied now
    const float gv = FZ ? g_value(gent, gbits) : __builtin_bit_cast(float, gbits);
    __syncthreads();
    apply_scales();
    if constexpr (EXTRA) {
      if (norm && !FZ) {  // 1 / sqrt(mean z^2 + eps)
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
    if constexpr (kXLds) {
      if (xlds) {
#pragma unroll
        for (int k = 0; k < kXPT; ++k) s_xu[threadIdx.x + k * kBlock] = xs[k];
      }
    }
    compact_segment(s_h, nrows, row0, seg, t, DENSE, act, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    LaneVec<W, CPLU, limb_vec<W, CPLU>()> xr;
    if constexpr (kXLds) {
      if (xlds) {
        dot_rows<W, CPLU, 2>(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, lpru, lpru_log2, s_cnt, xr, up_row,
                             up_sink, nullptr, s_xu);
        return;
      }
    }
    make_lane_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU>(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  } else {
    static_assert(CPLG == CPLU, "standard gating shares the x registers");
    if constexpr (!DENSE && !is_quant<W>()) {
      if (lpru == kWave) {  // one row a wave: the W_up rows join the gate stream
        __shared__ float s_zv[kSegMax];
        gate_up_stream<W, CPLU, FULL>(x, gate_w, w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, row0, nrows, t, form,
                                      s_h, s_zv);
        __syncthreads();
        compact_segment(s_h, nrows, row0, seg, t, false, act, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act,
                        s_zv, seg_zval);
        return;
      }
    }
    LaneVec<W, CPLU> xr;
    constexpr bool kLate = !is_quant<W>();
    if constexpr (!kLate) make_lane_vec<W, CPLU>(x, Cu, lane_id() & (lpru - 1), lpru, xr);
    dot_rows<W, CPLU, kLate>(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg, Cg, lprg, lprg_log2, nrows, xr, gate_row,
                             gate_sink, x);
    __syncthreads();
    apply_scales();
    compact_segment(s_h, nrows, row0, seg, t, DENSE, act, s_list, s_act, &s_cnt, seg_count, seg_idx, seg_act);
    __syncthreads();
    dot_rows<W, CPLU>(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu, Cu, lpru, lpru_log2, s_cnt, xr, up_row, up_sink);
  }
}

// y += sum over the listed neurons of a row chunk of zval * w_down_t[neuron], for one
// column slice of LG 16-byte chunks a row.  A listed neuron with zval exactly 0 (the
// s_gated site) is skipped: its row is not read.  Workgroup b covers column slice b % S of
// the neurons in segments [c nseg/R, (c+1) nseg/R), c = b / S.  A wave reads 64/LG rows an
// instruction (LG lanes a row: 32 for fp32 / bf16, whose 32 chunks are 512 bytes of a bf16
// row; 16 for the quantized formats, so that a slice stays 256 - 512 columns wide).  Each lane's
// partial sums go to LDS; the row groups and waves are added there in a fixed order, and
// one atomic per column adds them into y (y was cleared by the gate kernel).
//
// Every load is a raw buffer load (an unused slot gets an offset past the buffer), and
// every LDS read of the list is unconditional, so that the loads of a round issue back to
// back: with predicated loads each one sat behind its own branch and LDS wait.  The host
// guarantees w_down_t < 2^31 bytes.
constexpr int kDownSlotsPerThread = 8, kDownSlots = kDownSlotsPerThread * kBlock;

// The z slots of a single-token LoPA call whose gate kernel computed z: their tags go back to
// zero for the next call (the gate kernel, which read them, has finished).
__device__ __forceinline__ void clear_zslots(uint64_t* zslot, int n) {
  if (blockIdx.x == 0)
    for (int j = threadIdx.x; j < n; j += kBlock) zslot[j] = 0;
}

template <class W, bool DENSE, int LG>
__global__ __launch_bounds__(kBlock) void k_down_t1(const int32_t* __restrict__ seg_count,
                                                    const int32_t* __restrict__ seg_idx,
                                                    const float* __restrict__ seg_zval, int nseg, int d_ff, int R,
                                                    const uint4* __restrict__ w_down_t, int C, int d,
                                                    float* __restrict__ y, const float* __restrict__ s_down,
                                                    uint64_t* __restrict__ zslot, int nzclear) {
  constexpr int EPC = W::EPC, U = 8, kWaves = kBlock / kWave, RG = kWave / LG, PT = kDownSlotsPerThread;
  clear_zslots(zslot, nzclear);
  extern __shared__ int s_dyn[];  // the compacted list (sparse only): indices, then values
  __shared__ int s_cnt[kWave];
  __shared__ int s_off[kWave + 1];
  // [wave row group][e][q], rows padded to LG + 1: lanes (consecutive q) write, and
  // threads (consecutive e) read, distinct banks
  __shared__ float s_red[kWaves * RG][EPC * (LG + 1)];

  const int S = (C + LG - 1) / LG;
  const int chunk = blockIdx.x / S, slice = blockIdx.x % S;
  const Split chunks(nseg, R), segs(d_ff, nseg);
  const int seg_lo = chunks.start(chunk), seg_hi = chunks.start(chunk + 1);
  const int row_lo = segs.start(seg_lo), row_hi = segs.start(seg_hi);
  const int raw_n = row_hi - row_lo;
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const Buf zb = make_buf(seg_zval, 4u * (uint32_t)d_ff);

  int n = raw_n;
  int* l_idx = s_dyn;
  float* l_z = reinterpret_cast<float*>(s_dyn + raw_n);
  if constexpr (!DENSE) {
    // one round trip: the chunk's slots into registers (kDownSlots a round), the segment
    // counts into LDS; then each valid slot goes to its place in the compacted list
    const Buf ib = make_buf(seg_idx, 4u * (uint32_t)d_ff);
    for (int p0 = 0; p0 < raw_n; p0 += kDownSlots) {
      int ri[PT];
      float rz[PT];
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        const int p = p0 + threadIdx.x + u * kBlock;
        const uint32_t off = p < raw_n ? 4u * (uint32_t)(row_lo + p) : kOOB;
        ri[u] = ldb32(ib, off);
        rz[u] = __int_as_float(ldb32(zb, off));
      }
      if (p0 == 0 && wave == 0) {
        const int nsc = seg_hi - seg_lo;  // <= 64, guaranteed by the host
        const Buf cb = make_buf(seg_count, 4u * (uint32_t)nseg);
        const int c = ldb32(cb, lane < nsc ? 4u * (uint32_t)(seg_lo + lane) : kOOB);
        const int v = wave_inclusive_scan(c);
        s_cnt[lane] = c;
        s_off[lane] = v - c;
        if (lane == kWave - 1) s_off[kWave] = v;
      }
      __syncthreads();
      // segment and rank of each slot, their counts and offsets read back to back; a
      // group of slots wholly past the chunk is skipped (a workgroup-uniform test)
      int rw[PT], re[PT], rc[PT], ro[PT];
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        if (p0 + u * kBlock >= raw_n) break;
        const int p = p0 + threadIdx.x + u * kBlock;
        const int row = row_lo + (p < raw_n ? p : 0);
        rw[u] = segs.of(row) - seg_lo;
        re[u] = row - segs.start(seg_lo + rw[u]);
      }
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        if (p0 + u * kBlock >= raw_n) break;
        rc[u] = s_cnt[rw[u]];
        ro[u] = s_off[rw[u]];
      }
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        if (p0 + u * kBlock >= raw_n) break;
        if (p0 + threadIdx.x + u * kBlock < raw_n && re[u] < rc[u]) {
          l_idx[ro[u] + re[u]] = ri[u];
          l_z[ro[u] + re[u]] = rz[u];
        }
      }
    }
    __syncthreads();
    n = s_off[kWave];
  }

  const Buf wb = make_buf(w_down_t, 16u * (uint32_t)d_ff * (uint32_t)C);
  const Buf sb = make_buf(s_down, 4u * (uint32_t)d_ff);
  const int q = lane % LG, g = lane / LG;
  const int ch = slice * LG + q;
  const bool cvalid = ch < C;
  float acc[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
  // A round: U slots of each of the wave's row groups, rows kb + g + u kWaves RG (kb the
  // wave's first row, wave-uniform).  Two register sets alternate, so that the next round's
  // rows are in flight while a round is folded (a chunk of more rows than one round had
  // waited a whole round trip per round).  Rows past n load nothing and fold nothing.
  struct Round {
    uint4 wv[U];
    float zz[U], sc[U];
  };
  auto issue = [&](Round& rd, int kb) {
    int row[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = kb + g + u * kWaves * RG;
      ok[u] = kk < n;
      if constexpr (DENSE) {
        row[u] = row_lo + kk;
      } else {
        const int j = ok[u] ? kk : 0;  // n >= 1 here
        row[u] = l_idx[j];
        rd.zz[u] = ok[u] ? l_z[j] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (DENSE) rd.zz[u] = __int_as_float(ldb32(zb, ok[u] ? 4u * (uint32_t)row[u] : kOOB));
      // a zero gated value (the s_gated site) needs no W_down row
      const bool need = ok[u] && cvalid && (DENSE || rd.zz[u] != 0.f);
      rd.wv[u] = ldb_nt(wb, need ? 16u * ((uint32_t)row[u] * (uint32_t)C + (uint32_t)ch) : kOOB);
      if constexpr (is_quant<W>())  // the row's scale (0 for an unused slot)
        rd.sc[u] = __int_as_float(ldb32(sb, ok[u] ? 4u * (uint32_t)row[u] : kOOB));
    }
  };
  auto fold = [&](const Round& rd, int u) {
    float f[EPC];
    unpack(W{}, rd.wv[u], f);
    const float z = is_quant<W>() ? rd.zz[u] * rd.sc[u] : rd.zz[u];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = fmaf(z, f[e], acc[e]);
  };
  // A full round folds every slot.  A round with the wave's last row stops there (a
  // wave-uniform test): unpacking the empty slots costs up to 96 ALU ops a slot.  Both
  // branches use every load, so none of them is sunk behind a test.
  auto fold_round = [&](const Round& rd, int kb) {
    if (kb + (U - 1) * kWaves * RG < n) {
#pragma unroll
      for (int u = 0; u < U; ++u) fold(rd, u);
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (kb + u * kWaves * RG >= n) break;
        fold(rd, u);
      }
    }
  };
  constexpr int kStride = kWaves * RG * U;  // rows of one round of the workgroup
  if (wave * RG < n) {
    Round r0, r1;
    int kb = wave * RG;
    issue(r0, kb);
    issue_barrier();
    if (kb + kStride >= n) {
      fold_round(r0, kb);
    } else {
      for (;; kb += 2 * kStride) {
        issue(r1, kb + kStride);
        issue_barrier();
        fold_round(r0, kb);
        issue(r0, kb + 2 * kStride);
        issue_barrier();
        fold_round(r1, kb + kStride);
        if (kb + 2 * kStride >= n) break;
      }
    }
  }
#pragma unroll
  for (int e = 0; e < EPC; ++e) s_red[wave * RG + g][e * (LG + 1) + q] = acc[e];
  __syncthreads();
  // consecutive threads, consecutive columns: each atomic instruction covers whole lines
  for (int o = threadIdx.x; o < LG * EPC; o += kBlock) {
    const int qq = o / EPC, e = o - qq * EPC;
    float sum = s_red[0][e * (LG + 1) + qq];
#pragma unroll
    for (int w = 1; w < kWaves * RG; ++w) sum += s_red[w][e * (LG + 1) + qq];
    const int col = slice * LG * EPC + o;
    if (col < d) unsafeAtomicAdd(y + col, sum);
  }
}

// The same product for a batch of T tokens (up to kTokChunk), TG of them a workgroup
// (blockIdx.y picks the token group): every listed row of the chunk (a neuron active for
// any token of the batch) is read once per token group and folded into TG accumulator
// sets.  Zero gated values add nothing; a row whose values are all zero for the group is
// not read.  The lists and the group's gated values are staged in LDS as in the
// single-token kernel.
template <class W, bool DENSE, int LG, int TG>
__global__ __launch_bounds__(kBlock) void k_down_tb(const int32_t* __restrict__ seg_count,
                                                    const int32_t* __restrict__ seg_idx,
                                                    const float* __restrict__ seg_zval, int nseg, int d_ff, int R,
                                                    int slots, int T, const uint4* __restrict__ w_down_t, int C,
                                                    int d, float* __restrict__ y, const float* __restrict__ s_down) {
  constexpr int EPC = W::EPC, U = 8, kWaves = kBlock / kWave, RG = kWave / LG, PT = kDownSlotsPerThread;
  extern __shared__ int s_dyn[];  // the compacted list: row indices, then TG rows of gated values
  __shared__ int s_cnt[kWave];
  __shared__ int s_off[kWave + 1];
  __shared__ float s_red[kWaves * RG][EPC * (LG + 1)];

  const int S = (C + LG - 1) / LG;
  const int chunk = blockIdx.x / S, slice = blockIdx.x % S;
  const int t0 = blockIdx.y * TG, tn = min(TG, T - t0);
  const Split chunks(nseg, R), segs(d_ff, nseg);
  const int seg_lo = chunks.start(chunk), seg_hi = chunks.start(chunk + 1);
  const int row_lo = segs.start(seg_lo), row_hi = segs.start(seg_hi);
  const int raw_n = row_hi - row_lo;
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const Buf zb = make_buf(seg_zval, 4u * (uint32_t)slots * (uint32_t)T);
  int* l_idx = s_dyn;
  float* l_z = reinterpret_cast<float*>(s_dyn + raw_n);  // [TG][raw_n]

  int n = raw_n;
  {
    // one round trip: the chunk's slots and the group's gated values into registers, the
    // segment counts into LDS; then each valid slot goes to its place in the list
    const Buf ib = make_buf(seg_idx, 4u * (uint32_t)d_ff);
    for (int p0 = 0; p0 < raw_n; p0 += kDownSlots) {
      int ri[PT];
      float rz[PT][TG];
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        const int p = p0 + threadIdx.x + u * kBlock;
        const bool ok = p < raw_n;
        const uint32_t slot = (uint32_t)(row_lo + p);
        ri[u] = DENSE ? (int)slot : ldb32(ib, ok ? 4u * slot : kOOB);
#pragma unroll
        for (int v = 0; v < TG; ++v)
          rz[u][v] = __int_as_float(ldb32(zb, ok && v < tn ? 4u * ((uint32_t)(t0 + v) * (uint32_t)slots + slot) : kOOB));
      }
      if constexpr (!DENSE) {
        if (p0 == 0 && wave == 0) {
          const int nsc = seg_hi - seg_lo;  // <= 64, guaranteed by the host
          const Buf cb = make_buf(seg_count, 4u * (uint32_t)nseg);
          const int c = ldb32(cb, lane < nsc ? 4u * (uint32_t)(seg_lo + lane) : kOOB);
          const int v = wave_inclusive_scan(c);
          s_cnt[lane] = c;
          s_off[lane] = v - c;
          if (lane == kWave - 1) s_off[kWave] = v;
        }
        __syncthreads();
      }
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        const int p = p0 + threadIdx.x + u * kBlock;
        if (p0 + u * kBlock >= raw_n) break;
        int pos = p;
        bool keep = p < raw_n;
        if constexpr (!DENSE) {
          const int row = row_lo + (keep ? p : 0);
          const int w = segs.of(row) - seg_lo;
          const int e = row - segs.start(seg_lo + w);
          keep = keep && e < s_cnt[w];
          pos = s_off[w] + e;
        }
        if (keep) {
          l_idx[pos] = ri[u];
#pragma unroll
          for (int v = 0; v < TG; ++v) l_z[v * raw_n + pos] = rz[u][v];
        }
      }
    }
    __syncthreads();
    if constexpr (!DENSE) n = s_off[kWave];
  }

  const Buf wb = make_buf(w_down_t, 16u * (uint32_t)d_ff * (uint32_t)C);
  const Buf sb = make_buf(s_down, 4u * (uint32_t)d_ff);
  const int q = lane % LG, g = lane / LG;
  const int ch = slice * LG + q;
  const bool cvalid = ch < C;
  float acc[TG][EPC];
#pragma unroll
  for (int v = 0; v < TG; ++v)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[v][e] = 0.f;
  for (int kb = wave * RG; kb < n; kb += kWaves * RG * U) {
    uint4 wv[U];
    float zz[U][TG], sc[U];
    int row[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = kb + g + u * kWaves * RG;
      ok[u] = kk < n;
      const int j = ok[u] ? kk : 0;  // n >= 1 here
      row[u] = l_idx[j];
#pragma unroll
      for (int v = 0; v < TG; ++v) zz[u][v] = ok[u] ? l_z[v * raw_n + j] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bool any = false;
#pragma unroll
      for (int v = 0; v < TG; ++v) any = any || zz[u][v] != 0.f;
      const bool need = ok[u] && cvalid && (DENSE || any);
      wv[u] = ldb_nt(wb, need ? 16u * ((uint32_t)row[u] * (uint32_t)C + (uint32_t)ch) : kOOB);
      if constexpr (is_quant<W>()) sc[u] = __int_as_float(ldb32(sb, ok[u] ? 4u * (uint32_t)row[u] : kOOB));
    }
    issue_barrier();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kb + u * kWaves * RG >= n) break;  // past the wave's last row (wave-uniform)
      float f[EPC];
      unpack(W{}, wv[u], f);
#pragma unroll
      for (int v = 0; v < TG; ++v) {
        const float z = is_quant<W>() ? zz[u][v] * sc[u] : zz[u][v];
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[v][e] = fmaf(z, f[e], acc[v][e]);
      }
    }
  }
  // one token at a time through the LDS tile: the row groups and waves in a fixed order,
  // then one atomic per column (v runs to TG so that acc is indexed at compile time)
#pragma unroll
  for (int v = 0; v < TG; ++v) {
    if (v >= tn) break;  // workgroup-uniform
#pragma unroll
    for (int e = 0; e < EPC; ++e) s_red[wave * RG + g][e * (LG + 1) + q] = acc[v][e];
    __syncthreads();
    for (int o = threadIdx.x; o < LG * EPC; o += kBlock) {
      const int qq = o / EPC, e = o - qq * EPC;
      float sum = s_red[0][e * (LG + 1) + qq];
#pragma unroll
      for (int w = 1; w < kWaves * RG; ++w) sum += s_red[w][e * (LG + 1) + qq];
      const int col = slice * LG * EPC + o;
      if (col < d) unsafeAtomicAdd(y + (size_t)(t0 + v) * d + col, sum);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ generic kernels
// Any T <= kTokChunk, any d / d_ff / r, element-wise loads.  Used for shapes and
// batches the specialised kernels do not cover.
// <row `row` of a [rows][len] matrix, vec> for one wave (every lane gets the sum).
// Rows of whole 16-byte chunks are read a chunk a lane (raw buffer loads, UF chunks of
// a lane in flight together, the vector as float4); other rows element by element.
template <class W>
__device__ __forceinline__ float wave_row_dot(const void* __restrict__ mat, int row, int len,
                                              const float* __restrict__ vec) {
  constexpr int EPC = W::EPC, UF = 64 / EPC < 4 ? 64 / EPC : 4;
  const int lane = lane_id();
  float s = 0.f;
  if (len % EPC == 0) {
    const int C = len / EPC;
    const Buf rb = make_buf(static_cast<const char*>(mat) + (size_t)row * (size_t)C * 16u, 16u * (uint32_t)C);
    const Buf vb = make_buf(vec, 4u * (uint32_t)len);
    for (int c0 = 0; c0 < C; c0 += UF * kWave) {
      uint4 w[UF];
      uint4 xv[UF][EPC / 4];
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        const int ch = c0 + u * kWave + lane;
        const bool ok = ch < C;
        w[u] = ldb(rb, ok ? 16u * (uint32_t)ch : kOOB);
#pragma unroll
        for (int i = 0; i < EPC / 4; ++i) xv[u][i] = ldb(vb, ok ? 16u * (uint32_t)(ch * (EPC / 4) + i) : kOOB);
      }
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        float f[EPC];
        unpack(W{}, w[u], f);
#pragma unroll
        for (int i = 0; i < EPC / 4; ++i) {
          s = fmaf(f[4 * i], __uint_as_float(xv[u][i].x), s);
          s = fmaf(f[4 * i + 1], __uint_as_float(xv[u][i].y), s);
          s = fmaf(f[4 * i + 2], __uint_as_float(xv[u][i].z), s);
          s = fmaf(f[4 * i + 3], __uint_as_float(xv[u][i].w), s);
        }
      }
    }
  } else {
    for (int j = lane; j < len; j += kWave) s = fmaf(welem(W{}, mat, (size_t)row * len + j), vec[j], s);
  }
  return wave_sum(s);
}

// Token vectors staged in LDS by the element-wise gate kernel: at most kVecTok of them
// and kVecFloats floats in all.
constexpr int kVecTok = 4, kVecFloats = 8192;

// out[v] = <row `row` of a [rows][len] matrix, sv + v len> for v < tn <= kVecTok, the
// vectors in LDS; one wave, every lane gets the sums.  The lane's chunks of the row are
// loaded once for all the vectors.
template <class W>
__device__ __forceinline__ void wave_row_dots_lds(const void* __restrict__ mat, int row, int len, const float* sv,
                                                  int tn, float (&out)[kVecTok]) {
  constexpr int EPC = W::EPC, UF = 64 / EPC < 4 ? 64 / EPC : 4;
  const int lane = lane_id();
  float acc[kVecTok];
#pragma unroll
  for (int v = 0; v < kVecTok; ++v) acc[v] = 0.f;
  if (len % EPC == 0) {
    const int C = len / EPC;
    const Buf rb = make_buf(static_cast<const char*>(mat) + (size_t)row * (size_t)C * 16u, 16u * (uint32_t)C);
    for (int c0 = 0; c0 < C; c0 += UF * kWave) {
      uint4 w[UF];
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        const int ch = c0 + u * kWave + lane;
        w[u] = ldb(rb, ch < C ? 16u * (uint32_t)ch : kOOB);
      }
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        const int ch = c0 + u * kWave + lane;
        if (ch < C) {
          float f[EPC];
          unpack(W{}, w[u], f);
#pragma unroll
          for (int v = 0; v < kVecTok; ++v)
            if (v < tn) {
              const float4* xp = reinterpret_cast<const float4*>(sv + v * len + ch * EPC);
#pragma unroll
              for (int i = 0; i < EPC / 4; ++i) {
                const float4 xv = xp[i];
                acc[v] = fmaf(f[4 * i], xv.x, acc[v]);
                acc[v] = fmaf(f[4 * i + 1], xv.y, acc[v]);
                acc[v] = fmaf(f[4 * i + 2], xv.z, acc[v]);
                acc[v] = fmaf(f[4 * i + 3], xv.w, acc[v]);
              }
            }
        }
      }
    }
  } else {
    for (int j = lane; j < len; j += kWave) {
      const float wj = welem(W{}, mat, (size_t)row * len + j);
#pragma unroll
      for (int v = 0; v < kVecTok; ++v)
        if (v < tn) acc[v] = fmaf(wj, sv[v * len + j], acc[v]);
    }
  }
#pragma unroll
  for (int v = 0; v < kVecTok; ++v) out[v] = wave_sum(acc[v]);
}

template <class W>
__global__ __launch_bounds__(kBlock) void k_lopa_z_generic(const float* __restrict__ x, const void* __restrict__ A,
                                                           int T, int d, int r, float* __restrict__ z,
                                                           const float* __restrict__ s_a) {
  const int k = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
  if (k >= r) return;
  const int lane = lane_id();
  for (int tau = 0; tau < T; ++tau) {
    float s = wave_row_dot<W>(A, k, d, x + (size_t)tau * d);
    if constexpr (is_quant<W>()) s *= s_a[k];
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
                                                            Form form, const float* __restrict__ s_g,
                                                            const float* __restrict__ s_up) {
  __shared__ float s_h[kSegMax][kTokChunk];
  __shared__ int s_list[kSegMax];
  __shared__ int s_cnt;
  __shared__ __align__(16) float s_vec[kVecFloats];
  const int seg = blockIdx.x;
  const Split segs(d_ff, nseg);
  const int row0 = segs.start(seg), nrows = segs.start(seg + 1) - row0;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  constexpr int kWaves = kBlock / kWave;
  const int len = LOPA ? r : d;
  const float* vec = LOPA ? z : x;
  clear_output(y, T * d, meta, nseg);

  // rows `k` (k = wave, wave + 4, ... < n) dotted with every token's vector `v` (len
  // floats a token), the vectors staged in LDS a group of tokens at a time when they fit,
  // so that each row chunk is loaded once a group and the vectors come from LDS;
  // put(k, tau, value) takes the results
  auto rows_by_tokens = [&](const void* mat, auto row_of, int n, const float* v, int vlen, auto put) {
    const int tg = vlen <= kVecFloats ? min(kVecTok, kVecFloats / vlen) : 0;
    if (tg == 0) {  // too long for LDS: from memory, a token at a time
      for (int k = wave; k < n; k += kWaves)
        for (int tau = 0; tau < T; ++tau) put(k, tau, wave_row_dot<W>(mat, row_of(k), vlen, v + (size_t)tau * vlen));
      return;
    }
    for (int t0 = 0; t0 < T; t0 += tg) {
      const int tn = min(tg, T - t0);
      __syncthreads();  // the previous group's readers are done
      for (int i = threadIdx.x; i < tn * vlen; i += kBlock) s_vec[i] = v[(size_t)t0 * vlen + i];
      __syncthreads();
      for (int k = wave; k < n; k += kWaves) {
        float o[kVecTok];
        wave_row_dots_lds<W>(mat, row_of(k), vlen, s_vec, tn, o);
#pragma unroll
        for (int u = 0; u < kVecTok; ++u)
          if (u < tn) put(k, t0 + u, o[u]);
      }
    }
  };

  rows_by_tokens(
      gate_w, [&](int k) { return row0 + k; }, nrows, vec, len, [&](int k, int tau, float s) {
        if constexpr (is_quant<W>()) s *= s_g[row0 + k];
        if (lane == 0) s_h[k][tau] = s;
      });
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
  rows_by_tokens(
      w_up, [&](int e) { return row0 + s_list[e]; }, cnt, x, d, [&](int e, int tau, float s) {
        const int kr = s_list[e];
        if constexpr (is_quant<W>()) s *= s_up[row0 + kr];
        if (lane == 0) seg_zval[(size_t)tau * slots + row0 + e] = s_h[kr][tau] * (FULL ? up_value(form.silu_up, s) : s);
      });
}

// thread per output column; tokens in groups of 8 accumulators; y written directly
template <class W, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_down_generic(const int32_t* __restrict__ seg_count,
                                                         const int32_t* __restrict__ seg_idx,
                                                         const float* __restrict__ seg_zval, int nseg, int d_ff,
                                                         int slots, const void* __restrict__ w_down_t, int T, int d,
                                                         float* __restrict__ y, const float* __restrict__ s_down,
                                                         uint64_t* __restrict__ zslot, int nzclear) {
  extern __shared__ int s_pre[];  // [nseg + 1] list offsets (sparse only)
  clear_zslots(zslot, nzclear);
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
          float w = welem(W{}, w_down_t, (size_t)row * d + col);
          if constexpr (is_quant<W>()) w *= s_down[row];
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

// chunks a lane holds of a vector of C chunks: `lo` if 64 lanes cover it so, else 2 lo,
// else 0 (too long for the single-token kernels)
int cpl_pick(int C, int lo) { return C <= lo * kWave ? lo : (C <= 2 * lo * kWave ? 2 * lo : 0); }
// the smaller choice per format: 16-byte chunks hold 4 to 32 elements, and the quantized
// formats keep their vector as limbs (3 or 6 words per 4 words of codes)
template <class W>
constexpr int cpl_lo() {
  if constexpr (is_quant<W>())
    return W::LB == 8 ? 4 : 2;
  else
    return 8;
}
int cpl_for(int C) { return cpl_pick(C, 8); }
// bytes of a rows x cols matrix in format wdt
int64_t mat_bytes(int wdt, int64_t rows, int64_t cols) {
  return wdt == 0 ? 4 * rows * cols : wdt == 1 ? 2 * rows * cols : wdt == 2 ? rows * cols : rows * (cols / 2);
}
int epc_of(int wdt) { return wdt == 0 ? WF32::EPC : wdt == 1 ? WBf16::EPC : wdt == 2 ? WI8::EPC : WI4::EPC; }
int cpl_lo_of(int wdt) { return wdt == 0 ? cpl_lo<WF32>() : wdt == 1 ? cpl_lo<WBf16>() : wdt == 2 ? cpl_lo<WI8>() : cpl_lo<WI4>(); }

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

// At least kSegMinRows rows a segment, and at most d / kDnChunkCapDiv row chunks in the down
// kernel: on a small FFN (d 256, d_ff 1024) one-row segments over 768 workgroups and 256 row
// chunks, each chunk adding into the same few cache lines of y, left the call at 13.3 us; with
// both limits it takes 7.8 us.  The 8B and 70B shapes are above both limits.
constexpr int kSegMinRows = 16;
constexpr int kDnChunkCapDiv = 16;

// Segments for the T = 1 gate kernel: one row-balanced segment per workgroup slot the
// GPU holds at once (so every CU gets the same number of rows; more segments than
// resident slots measured slower), never more than kSegMax rows per segment nor fewer than
// kSegMinRows (where d_ff allows).  `per_cu` caches the kernel's occupancy.
template <class K>
int resident_segments(K kernel, int* per_cu, int d_ff) {
  if (*per_cu == 0) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, 0) != hipSuccess || n <= 0) n = 1;
    *per_cu = n;
  }
  int g = cu_count() * *per_cu;
  const int lo = (d_ff + kSegMax - 1) / kSegMax;
  const int hi = (d_ff + kSegMinRows - 1) / kSegMinRows;
  if (g > hi) g = hi;
  if (g < lo) g = lo;
  if (g > d_ff) g = d_ff;
  return g;
}

// The fast single-token kernels address a matrix with 32-bit byte offsets below 2^31.
bool fast_ok(const Shape& sh, Gate g) {
  const int epc_ = epc_of(sh.wdt), lo = cpl_lo_of(sh.wdt);
  const int64_t lim = int64_t(1) << 31;
  if (sh.T != 1 || sh.d % epc_ != 0 || cpl_pick(sh.d / epc_, lo) == 0) return false;
  if (mat_bytes(sh.wdt, sh.d_ff, sh.d) >= lim) return false;
  if (g == Gate::LoPA && (sh.r % epc_ != 0 || cpl_pick(sh.r / epc_, lo) == 0 ||
                          mat_bytes(sh.wdt, sh.r, sh.d) >= lim || mat_bytes(sh.wdt, sh.d_ff, sh.r) >= lim))
    return false;
  return true;
}

template <class W, bool LOPA, bool DENSE, int FORM, int CPLG, int CPLU, int CPLA = 0>
hipError_t go_gate_up_t1(const Shape& sh, const Form& form, const float* x, const void* gate_w, const void* w_up,
                         float t, Workspace& ws, float* y, hipStream_t s, const void* lopa_a = nullptr) {
  const int Cu = sh.d / W::EPC, Cg = LOPA ? sh.r / W::EPC : Cu;
  const int lpru = lanes_per_row(Cu, CPLU), lprg = lanes_per_row(Cg, CPLG);
  auto kernel = k_gate_up_t1<W, LOPA, DENSE, CPLG, CPLU, FORM, CPLA>;
  static int per_cu = 0;  // one cache per instantiation
  ws.nseg = resident_segments(kernel, &per_cu, sh.d_ff);
  return launch_gate_kernel(kernel, ws.nseg, s, x, (const float*)ws.z, static_cast<const uint4*>(gate_w), Cg, lprg,
                            ilog2(lprg), static_cast<const uint4*>(w_up), Cu, lpru, ilog2(lpru), sh.d_ff, ws.nseg, t,
                            ws.meta, ws.seg_count, ws.seg_idx, ws.seg_act, ws.seg_zval, y, sh.d, form,
                            (const float*)ws.zsq, (const float*)ws.gx, LOPA ? sh.sc.b : sh.sc.gate, sh.sc.up,
                            static_cast<const uint4*>(lopa_a), ws.zslot);
}

// Whether the single-token LoPA gate kernel computes z itself: fp32 / bf16 rows whose B rows
// take at most the lower chunk count a lane (z staged in LDS), and r within kFusedZMax.
template <class W>
bool fuses_z(const Shape& sh) {
  if constexpr (is_quant<W>()) {
    return false;
  } else {
    return sh.T == 1 && sh.r >= 1 && sh.r <= kFusedZMax && fast_ok(sh, Gate::LoPA) &&
           cpl_pick(sh.r / W::EPC, cpl_lo<W>()) == cpl_lo<W>();
  }
}

template <class W, bool LOPA, bool DENSE, int FORM>
hipError_t gate_up_fast(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up, float t,
                        Workspace& ws, float* y, hipStream_t s, const void* lopa_a) {
  constexpr int L = cpl_lo<W>(), H = 2 * L;
  const int cplu = cpl_pick(sh.d / W::EPC, L);
  if constexpr (LOPA) {
    const int cplg = cpl_pick(sh.r / W::EPC, L);
    if constexpr (!is_quant<W>()) {
      // z computed in the gate kernel: an A row's chunks spread over the 256 threads, 2 a
      // thread while the row fits (rows of up to 512 chunks), else 4
      if (lopa_a && fuses_z<W>(sh)) {
        if (cplu == L)
          return go_gate_up_t1<W, true, DENSE, FORM, L, L, 2>(sh, f, x, gate_w, w_up, t, ws, y, s, lopa_a);
        return go_gate_up_t1<W, true, DENSE, FORM, L, H, 4>(sh, f, x, gate_w, w_up, t, ws, y, s, lopa_a);
      }
    }
    if (cplg == L && cplu == L) return go_gate_up_t1<W, true, DENSE, FORM, L, L>(sh, f, x, gate_w, w_up, t, ws, y, s);
    if (cplg == L && cplu == H) return go_gate_up_t1<W, true, DENSE, FORM, L, H>(sh, f, x, gate_w, w_up, t, ws, y, s);
    if (cplg == H && cplu == L) return go_gate_up_t1<W, true, DENSE, FORM, H, L>(sh, f, x, gate_w, w_up, t, ws, y, s);
    return go_gate_up_t1<W, true, DENSE, FORM, H, H>(sh, f, x, gate_w, w_up, t, ws, y, s);
  } else {
    if (cplu == L) return go_gate_up_t1<W, false, DENSE, FORM, L, L>(sh, f, x, gate_w, w_up, t, ws, y, s);
    return go_gate_up_t1<W, false, DENSE, FORM, H, H>(sh, f, x, gate_w, w_up, t, ws, y, s);
  }
}

template <class W, bool LOPA, bool DENSE, bool FULL>
hipError_t gate_up_generic(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up,
                           float t, Workspace& ws, float* y, hipStream_t s) {
  ws.nseg = (sh.d_ff + kSegGeneric - 1) / kSegGeneric;
  return launch_gate_kernel(k_gate_up_generic<W, LOPA, DENSE, FULL>, ws.nseg, s, x, (const float*)ws.z, gate_w, w_up,
                            sh.T, sh.d, sh.d_ff, sh.r, ws.nseg, t, ws.slots, ws.meta, ws.seg_count, ws.seg_idx,
                            ws.seg_act, ws.seg_zval, y, f, LOPA ? sh.sc.b : sh.sc.gate, sh.sc.up);
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

template <class W, int CPL>
void launch_z_row(const Shape& sh, const Form& form, const float* x, const void* A, const Workspace& ws,
                  hipStream_t s) {
  const GWork gw{form, x, ws.gx, 1, sh.d, sh.d_ff, sh.r};
  const int g = sh.r + (form.g_idx ? (g_items(sh.d_ff, 1) + kBlock - 1) / kBlock : 0);
  const int C = sh.d / W::EPC;
  const uint4* a = static_cast<const uint4*>(A);
  if (form.rms_eps > 0.f)
    k_lopa_z_row<W, CPL, true><<<g, kBlock, 0, s>>>(x, a, C, sh.r, ws.z, form.rms_gain, ws.zsq, gw);
  else
    k_lopa_z_row<W, CPL, false><<<g, kBlock, 0, s>>>(x, a, C, sh.r, ws.z, nullptr, nullptr, gw);
}

template <class W>
hipError_t lopa_z(const Shape& sh, const Form& form, const float* x, const void* A, const Workspace& ws,
                  hipStream_t s) {
  // one row a workgroup when the one-row-a-wave kernel (four rows a workgroup) would leave
  // compute units idle (measured: 8B r = 512, 4.0 -> 3.7 us; at 70B r = 1024, where the
  // latter fills the GPU, the row kernel took 6.2 us against 5.7)
  if constexpr (!is_quant<W>()) {
    const int C = sh.d / W::EPC;
    if (fast_ok(sh, Gate::LoPA) && C <= 8 * kBlock && sh.r < (kBlock / kWave) * cu_count()) {
      if (C <= kBlock)
        launch_z_row<W, 1>(sh, form, x, A, ws, s);
      else if (C <= 2 * kBlock)
        launch_z_row<W, 2>(sh, form, x, A, ws, s);
      else if (C <= 4 * kBlock)
        launch_z_row<W, 4>(sh, form, x, A, ws, s);
      else
        launch_z_row<W, 8>(sh, form, x, A, ws, s);
      return hipGetLastError();
    }
  }
  if (fast_ok(sh, Gate::LoPA)) {
    constexpr int L = cpl_lo<W>(), H = 2 * L;
    const int C = sh.d / W::EPC;
    const int cpl = cpl_pick(C, L), lpr = lanes_per_row(C, cpl), lg = ilog2(lpr);
    const int rows_per_block = (kBlock / kWave) * (kWave >> lg);
    const int grid = (sh.r + rows_per_block - 1) / rows_per_block;
    const uint4* a = static_cast<const uint4*>(A);
    const bool norm = form.rms_eps > 0.f;
    // with G, extra workgroups write G x for the gate kernel
    const GWork gw{form, x, ws.gx, 1, sh.d, sh.d_ff, grid};
    const int g = grid + (form.g_idx ? (g_items(sh.d_ff, 1) + kBlock - 1) / kBlock : 0);
    const float* gain = norm ? form.rms_gain : nullptr;
    float* zsq = norm ? ws.zsq : nullptr;
    if (cpl == L && norm)
      k_lopa_z_t1<W, L, true><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, gain, zsq, gw, sh.sc.a);
    else if (cpl == L)
      k_lopa_z_t1<W, L, false><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, gain, zsq, gw, sh.sc.a);
    else if (norm)
      k_lopa_z_t1<W, H, true><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, gain, zsq, gw, sh.sc.a);
    else
      k_lopa_z_t1<W, H, false><<<g, kBlock, 0, s>>>(x, a, C, lpr, lg, sh.r, ws.z, gain, zsq, gw, sh.sc.a);
  } else {
    const int grid = (sh.r + kBlock / kWave - 1) / (kBlock / kWave);
    k_lopa_z_generic<W><<<grid, kBlock, 0, s>>>(x, A, sh.T, sh.d, sh.r, ws.z, sh.sc.a);
  }
  return hipGetLastError();
}

// Down-projection grid for T = 1: S column slices x R row chunks, about wg_per_cu
// workgroups per CU, at most 64 segments per chunk.
void down_grid(int C, int lg, int wg_per_cu, int nseg, int d_ff, int d, int* S, int* R, size_t* shmem_rows) {
  *S = (C + lg - 1) / lg;
  int r = (wg_per_cu * cu_count() + *S - 1) / *S;
  if (r > d / kDnChunkCapDiv) r = d / kDnChunkCapDiv > 1 ? d / kDnChunkCapDiv : 1;
  const int rmin = (nseg + kWave - 1) / kWave;
  if (r < rmin) r = rmin;
  if (r > nseg) r = nseg;
  *R = r;
  // largest row range of a chunk: ceil(nseg / R) segments of at most ceil(d_ff / nseg) rows
  *shmem_rows = (size_t)((nseg + r - 1) / r) * (size_t)((d_ff + nseg - 1) / nseg);
}

template <class W, bool DENSE>
hipError_t down(const Shape& sh, const void* w_down_t, const Workspace& ws, float* y, hipStream_t s, int nzclear) {
  // lanes a row and workgroups per CU, as measured best on the 8B shape: a bf16 slice of
  // 512 columns at two workgroups per CU; int8 / int4 slices of 256 / 512 columns at one
  constexpr int LG = is_quant<W>() ? 16 : 32, WG_PER_CU = is_quant<W>() ? 1 : 2;
  // batches: TG tokens a workgroup (at most 64 accumulators a lane)
  constexpr int TG = 64 / W::EPC < 4 ? 64 / W::EPC : 4;
  const bool rows_ok = sh.d % W::EPC == 0 && mat_bytes(sh.wdt, sh.d_ff, sh.d) < (int64_t(1) << 31);
  const int C = sh.d / W::EPC;
  int S = 0, R = 0;
  size_t rows = 0;
  if (rows_ok) down_grid(C, LG, WG_PER_CU, ws.nseg, sh.d_ff, sh.d, &S, &R, &rows);
  const size_t shmem_t1 = DENSE ? 0 : 2 * sizeof(int) * rows, shmem_tb = (1 + TG) * sizeof(int) * rows;
  // bf16 rows of 1024 chunks or more (d >= 8192): 1 KB column slices, so that each workgroup
  // stages half as many slots (70B: 12.6 -> 12.2 us; on d = 4096 the 512-byte slices are faster)
  if constexpr (W::EPC == 8) {
    if (rows_ok && sh.T == 1 && C >= 1024) {
      int S2 = 0, R2 = 0;
      size_t rows2 = 0;
      down_grid(C, 64, WG_PER_CU, ws.nseg, sh.d_ff, sh.d, &S2, &R2, &rows2);
      const size_t shmem2 = DENSE ? 0 : 2 * sizeof(int) * rows2;
      if (shmem2 <= 96 * 1024) {
        k_down_t1<W, DENSE, 64><<<S2 * R2, kBlock, shmem2, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg,
                                                                 sh.d_ff, R2, static_cast<const uint4*>(w_down_t), C,
                                                                 sh.d, y, sh.sc.down, ws.zslot, nzclear);
        return hipGetLastError();
      }
    }
  }
  if (rows_ok && sh.T == 1 && shmem_t1 <= 96 * 1024) {
    k_down_t1<W, DENSE, LG><<<S * R, kBlock, shmem_t1, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff,
                                                             R, static_cast<const uint4*>(w_down_t), C, sh.d, y,
                                                             sh.sc.down, ws.zslot, nzclear);
  } else if (rows_ok && sh.T > 1 && shmem_tb <= 96 * 1024 && (int64_t)sh.T * ws.slots < (int64_t(1) << 29)) {
    const dim3 grid(S * R, (sh.T + TG - 1) / TG);
    k_down_tb<W, DENSE, LG, TG><<<grid, kBlock, shmem_tb, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg,
                                                               sh.d_ff, R, ws.slots, sh.T,
                                                               static_cast<const uint4*>(w_down_t), C, sh.d, y,
                                                               sh.sc.down);
  } else {
    const size_t shmem = DENSE ? 0 : sizeof(int) * (size_t)(ws.nseg + 1);
    const int grid = (sh.d + kBlock - 1) / kBlock;
    k_down_generic<W, DENSE><<<grid, kBlock, shmem, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff,
                                                        ws.slots, w_down_t, sh.T, sh.d, y, sh.sc.down, ws.zslot,
                                                        nzclear);
  }
  return hipGetLastError();
}

// the kernels for the form: the compile-time kind of the single-token kernel, the full
// flag of the element-wise one (G and the norm need LoPA; the options check enforces it)
template <class W, bool LOPA, bool DENSE>
hipError_t gate_up_form(const Shape& sh, bool fast, const Form& f, const float* x, const void* gate_w,
                        const void* w_up, float t, Workspace& ws, float* y, hipStream_t s, const void* lopa_a) {
  if (!fast)
    return f.full() ? gate_up_generic<W, LOPA, DENSE, true>(sh, f, x, gate_w, w_up, t, ws, y, s)
                    : gate_up_generic<W, LOPA, DENSE, false>(sh, f, x, gate_w, w_up, t, ws, y, s);
  if constexpr (LOPA)
    if (f.kind() == kFormLoPA)
      return gate_up_fast<W, LOPA, DENSE, kFormLoPA>(sh, f, x, gate_w, w_up, t, ws, y, s, lopa_a);
  return f.full() ? gate_up_fast<W, LOPA, DENSE, kFormAct>(sh, f, x, gate_w, w_up, t, ws, y, s, lopa_a)
                  : gate_up_fast<W, LOPA, DENSE, kFormDefault>(sh, f, x, gate_w, w_up, t, ws, y, s, lopa_a);
}

}  // namespace

// ------------------------------------------------------------------ launchers
hipError_t launch_rms_norm(float* z, int parts, int tc, int T, int r, const float* gain, float eps, hipStream_t s) {
  k_rms_norm<<<T, kBlock, 0, s>>>(z, parts, tc, r, gain, eps);
  return hipGetLastError();
}

// calls f with a value of the weight-format type of wdt
template <class F>
hipError_t by_format(int wdt, F&& f) {
  switch (wdt) {
    case 0: return f(WF32{});
    case 1: return f(WBf16{});
    case 2: return f(WI8{});
    default: return f(WI4{});
  }
}

hipError_t launch_lopa_z(const Shape& sh, const Form& form, const float* x, const void* lopa_a, const Workspace& ws,
                         hipStream_t s) {
  return by_format(sh.wdt, [&](auto w) { return lopa_z<decltype(w)>(sh, form, x, lopa_a, ws, s); });
}

bool lopa_fuses_z(const Shape& sh, const Form&) {
  return by_format(sh.wdt, [&](auto w) { return fuses_z<decltype(w)>(sh) ? hipSuccess : hipErrorNotSupported; }) ==
         hipSuccess;
}

hipError_t launch_gate_up(const Shape& sh, Gate g, bool dense, const Form& form, const float* x, const void* gate_w,
                          const void* w_up, float t, Workspace& ws, float* y, hipStream_t s, const void* lopa_a) {
  const bool lopa = g == Gate::LoPA;
  const bool fast = fast_ok(sh, g);
  if (lopa && !fast && form.rms_eps > 0.f) {  // the single-token kernel normalises z itself
    const hipError_t e = launch_rms_norm(ws.z, 1, ws.tc, sh.T, sh.r, form.rms_gain, form.rms_eps, s);
    if (e != hipSuccess) return e;
  }
  return by_format(sh.wdt, [&](auto w) {
    using W = decltype(w);
    if (lopa) return dense ? gate_up_form<W, true, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s, lopa_a)
                           : gate_up_form<W, true, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s, lopa_a);
    return dense ? gate_up_form<W, false, true>(sh, fast, form, x, gate_w, w_up, t, ws, y, s, nullptr)
                 : gate_up_form<W, false, false>(sh, fast, form, x, gate_w, w_up, t, ws, y, s, nullptr);
  });
}

hipError_t launch_down(const Shape& sh, bool dense, const void* w_down_t, const Workspace& ws, float* y,
                       hipStream_t s, bool clear_zslots) {
  const int nz = clear_zslots ? sh.r : 0;
  return by_format(sh.wdt, [&](auto w) {
    using W = decltype(w);
    return dense ? down<W, true>(sh, w_down_t, ws, y, s, nz) : down<W, false>(sh, w_down_t, ws, y, s, nz);
  });
}

}  // namespace ffn

// gfx950 kernels for a batch of 2..64 tokens with bf16 weights (paper Section 5.3: the
// rows of W_up / W_down are read once for the union of the tokens' active sets).
//
// Every contraction runs on the matrix cores (v_mfma_f32_16x16x32_bf16): LoPA's A x,
// the gate (W_gate x, or B z), the W_up dots of the union rows and the down
// projection.  Token-side operands (x, z, zval) enter as bf16 hi + lo pairs (v - hi
// rounded again): two MFMAs per step whose products are exact in fp32, so the split
// leaves a relative error of about 2^-16 per element, far inside the 1e-3 band of the
// active-set decision.  A 16-row weight tile is the A operand: lane l holds 8
// consecutive bf16 of row l mod 16 and the four lane groups l / 16 hold four
// consecutive 16-byte chunks.  Which k positions a lane group holds does not matter for
// a full reduction as long as both operands use the same ones.  Weights are read row by
// row (up to 256 contiguous bytes of a row per instruction) and reshaped into that
// layout through a wave-private LDS tile (see the streaming core).
//
// One call is three kernels (two for standard gating), one more above 16 tokens:
//   k_split_tokens (more than 16 tokens) the tokens split once into bf16 hi / lo planes
//                  in fragment order, read by the next two kernels;
//   k_lopa_z_mfma  z = A x as two partial sums over halves of the d range;
//   k_gate_up_mfma per segment of at most 64 rows: gate, union of the tokens' active rows,
//                  ascending, W_up dots of the union rows; zval = act * v is left in
//                  the A-operand fragment order of the down product (k_gate_up_q4 does the
//                  same for 2..4 tokens on 4x4x4 products, k_gate_up_mfma2 at two
//                  workgroups a CU where d_ff is large);
//   k_down_mfma    Y[tokens][cols] += Z[tokens][entries] D[entries][cols] over the
//                  union rows, segment by segment.
// A wave of the gate kernel multiplies four row tiles over a quarter of the k range, so
// each token fragment it loads (and splits, when it reads fp32 rows) feeds four tiles;
// the loads of the next k steps are in flight while the current ones are multiplied.  All operand loads are
// raw buffer loads: a lane with nothing to load (a row past the segment or the union,
// a token past the batch, a k step past the row) uses an offset beyond the buffer,
// which returns zero without a memory access, so every wave issues the same loads in
// the same order and the load counter waits stay exact.
//
// The down product needs, per lane, 8 entries of one column as the B operand, while a
// row gather gives a lane 8 columns of one entry.  The gathered rows go to LDS as they
// are and come back through gfx950's transposing LDS read (ds_read_b64_tr_b16), which
// exchanges 16-bit elements between the lanes of a 16-lane group: one pair of such
// reads hands every lane its 8 entries of one column.
#include "ffn_device.h"
#include "ffn_internal.h"

namespace ffn {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short short4_t __attribute__((ext_vector_type(4)));

constexpr int kTiles = 4;                // 16-row tiles of a gate segment
constexpr int kSegRowsB = 16 * kTiles;   // rows per gate segment (one 64-lane ballot)
constexpr int kParts = kBlock / kWave;   // k parts of a workgroup, one per wave
constexpr int kSegGrid = 256;            // most workgroups of the gate kernel, one per CU
constexpr int kSegGrid2 = 512;           // the same at two workgroups per CU

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8_t bf8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// v = hi + lo with both in bf16 (round to nearest even twice)
__device__ __forceinline__ void split8(const float (&v)[8], bf16x8_t& hi, bf16x8_t& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const __bf16 h = (__bf16)v[j];
    hi[j] = h;
    lo[j] = (__bf16)(v[j] - (float)h);
  }
}

// Chunk j (elements 8j .. 8j + 7) of a loaded 16-byte chunk of W, as 8 bf16: the chunk
// itself for bf16, the codes converted for int8 / int4 (exact: small integers), so that
// quantized rows enter the same bf16 operand tiles.  The row scales are applied to the
// products.
template <class W, int J>
__device__ __forceinline__ uint4 bf16_chunk(const uint4& v) {
  if constexpr (W::EPC == 8) {
    return v;
  } else {
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      float a, b;  // elements 8J + 2p and 8J + 2p + 1
      if constexpr (W::EPC == 16) {
        const uint32_t w = d[2 * J + (p >> 1)];
        const int e = 2 * (p & 1);
        a = (float)((int32_t)(w << (24 - 8 * e)) >> 24);
        b = (float)((int32_t)(w << (16 - 8 * e)) >> 24);
      } else {
        const uint32_t w = d[J];
        a = (float)((int32_t)(w << (28 - 8 * p)) >> 28);
        b = (float)((int32_t)(w << (24 - 8 * p)) >> 28);
      }
      // the high halves of both (selector bytes 2, 3 of the second operand, then of the first)
      o[p] = __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }
}
// all W::EPC / 8 of them into consecutive 16-byte slots of an LDS row
template <class W>
__device__ __forceinline__ void put_bf16_chunks(uint4* dst, const uint4& v) {
  dst[0] = bf16_chunk<W, 0>(v);
  if constexpr (W::EPC >= 16) dst[1] = bf16_chunk<W, 1>(v);
  if constexpr (W::EPC >= 32) {
    dst[2] = bf16_chunk<W, 2>(v);
    dst[3] = bf16_chunk<W, 3>(v);
  }
}

// k-step range [ks0, ks1) of k part kp out of np for rows of C chunks (4 chunks a step)
__device__ __forceinline__ void kpart(int C, int kp, int np, int* ks0, int* ks1) {
  const int nks = (C + 3) / 4;
  const int per = (nks + np - 1) / np;
  *ks0 = min(nks, kp * per);
  *ks1 = min(nks, *ks0 + per);
}

// ------------------------------------------------------------------ streaming core
// A group of KU consecutive k steps covers 16 RT weight rows x 4 KU chunks.  The group
// is read row by row, LPR = 4 KU lanes per row and 64 / LPR rows per instruction (256
// contiguous bytes per row for KU = 4), streamed past the caches, and reshaped into MFMA
// operands through a wave-private LDS tile: row br of the group sits at br * PITCH, one
// pad chunk per row keeping the operand reads free of bank conflicts.  (Loading the
// operand layout directly reads 64 bytes of each of 16 rows per instruction, which
// streams about 25% slower.)
// Quantized rows (W = WI8 / WI4): a loaded 16-byte chunk holds R8 = 2 or 4 of the tile's
// 8-element chunks, so a row takes 4 KU / R8 lanes; the codes are converted to bf16 as
// they go to the tile, which keeps the bf16 layout.
template <int RT, int KU, class W = WBf16>
struct WStage {
  static constexpr int R8 = W::EPC / 8;       // tile chunks per loaded chunk
  static constexpr int LPR = 4 * KU / R8;     // lanes per row of a load instruction
  static constexpr int RPI = kWave / LPR;     // rows per load instruction
  static constexpr int NI = (16 * RT + RPI - 1) / RPI;  // load instructions per group
  static constexpr int PITCH = 4 * KU + 1;    // 16-byte (8 bf16) chunks per LDS row
  static constexpr int WORDS = 16 * RT * PITCH;  // uint4 of one wave's tile
};

// Rows of this lane's load instructions: roff[i] = row_of(i RPI + lane / LPR) times the
// row's loaded chunks (C / R8 for rows of C tile chunks), or -1 where row_of gives no row
// (-1) or the lane falls past the tile's 16 RT rows.
template <int RT, int KU, class W = WBf16, class RowOf>
__device__ __forceinline__ void stage_rows(int* roff, int C, RowOf row_of) {  // roff: WStage::NI entries
  using S = WStage<RT, KU, W>;
  const int lane = lane_id();
#pragma unroll
  for (int i = 0; i < S::NI; ++i) {
    const int br = i * S::RPI + lane / S::LPR;
    const int r = br < 16 * RT ? row_of(br) : -1;
    roff[i] = r >= 0 ? r * (C / S::R8) : -1;
  }
}

// Operands of one group: the weight chunks as loaded and, per k step and token tile, the
// token fragment.  Two forms of the token side:
//  - fp32 rows: the 8 fp32 of the chunk (two 16-byte halves) from each of NP partial
//    copies of the token matrix, summed and split into hi / lo when multiplied.  A token
//    matrix is [T][8 C] fp32; partial copy p starts part_bytes * p into its buffer; tn = T.
//  - PRE (pre-split, NP = 1): b[u][nt][0] = the hi and lo fragments of the lane, read from
//    planes [k step][token tile][lane] of uint4 (k_split_tokens); the lo plane starts
//    part_bytes after the hi plane; tn = the planes' token-tile count.
template <int RT, int NT, int KU, int NP, class W = WBf16>
struct Frags {
  uint4 a[WStage<RT, KU, W>::NI];
  uint4 b[KU][NT][NP][2];
};

template <int RT, int NT, int KU, int NP, bool PRE = false, class W = WBf16>
__device__ __forceinline__ void load_frags(Frags<RT, NT, KU, NP, W>& f, const Buf& wb, int C,
                                           const int* roff, const Buf& tb, uint32_t part_bytes, int tn, int ks,
                                           int ks1) {
  using S = WStage<RT, KU, W>;
  const int lane = lane_id(), m = lane & 15, g = lane >> 4;
  {
    // the lane's loaded chunk gc of the group: tile chunks R8 gc .. R8 gc + R8 - 1
    const int gc = lane % S::LPR, c = 4 * ks / S::R8 + gc;
    const bool cv = ks + (gc * S::R8 >> 2) < ks1 && c < C / S::R8;
#pragma unroll
    for (int i = 0; i < S::NI; ++i)
      f.a[i] = ldb_nt(wb, (cv && roff[i] >= 0) ? 16u * (uint32_t)(roff[i] + c) : kOOB);
  }
  if constexpr (PRE) {
    static_assert(NP == 1, "pre-split tokens have one copy");
#pragma unroll
    for (int u = 0; u < KU; ++u)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const uint32_t off = ks + u < ks1 ? 16u * ((uint32_t)((ks + u) * tn + nt) * kWave + lane) : kOOB;
        f.b[u][nt][0][0] = ldb(tb, off);
        f.b[u][nt][0][1] = ldb(tb, off + part_bytes);
      }
    return;
  }
  const int T = tn;
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const int c = 4 * (ks + u) + g;
    const bool cv = ks + u < ks1 && c < C;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int tok = 16 * nt + m;
      const uint32_t off = (cv && tok < T) ? 32u * (uint32_t)(tok * C + c) : kOOB;
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        f.b[u][nt][p][0] = ldb(tb, off + p * part_bytes);
        f.b[u][nt][p][1] = ldb(tb, off + p * part_bytes + 16);
      }
    }
  }
}

// tile: this wave's LDS tile (Stage::WORDS uint4).  Every row tile is multiplied: one
// past the rows in use was loaded as zeros and only adds zeros to an accumulator that
// is never read.
// The token fragment of one k step and token tile from fp32 rows: the NP copies of the
// lane's 8 values summed, then split into hi / lo.
template <int NP>
__device__ __forceinline__ void sum_split(const uint4 (&b)[NP][2], bf16x8_t& hi, bf16x8_t& lo) {
  float v[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint4 q = b[0][h];
    v[4 * h] = __uint_as_float(q.x);
    v[4 * h + 1] = __uint_as_float(q.y);
    v[4 * h + 2] = __uint_as_float(q.z);
    v[4 * h + 3] = __uint_as_float(q.w);
  }
#pragma unroll
  for (int p = 1; p < NP; ++p)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint4 q = b[p][h];
      v[4 * h] += __uint_as_float(q.x);
      v[4 * h + 1] += __uint_as_float(q.y);
      v[4 * h + 2] += __uint_as_float(q.z);
      v[4 * h + 3] += __uint_as_float(q.w);
    }
  split8(v, hi, lo);
}

template <int RT, int NT, int KU, int NP, bool PRE = false, class W = WBf16>
__device__ __forceinline__ void mma_frags(const Frags<RT, NT, KU, NP, W>& f, uint4* tile, f32x4_t (&acc)[RT][NT]) {
  using S = WStage<RT, KU, W>;
  const int lane = lane_id(), m = lane & 15, g = lane >> 4;
#pragma unroll
  for (int i = 0; i < S::NI; ++i) {
    const int br = i * S::RPI + lane / S::LPR;
    if constexpr (S::R8 == 1) {
      tile[br * S::PITCH + lane % S::LPR] = f.a[i];
    } else if (br < 16 * RT) {  // lanes past the tile's rows loaded nothing
      put_bf16_chunks<W>(tile + br * S::PITCH + (lane % S::LPR) * S::R8, f.a[i]);
    }
  }
  __builtin_amdgcn_wave_barrier();  // LDS operations of a wave complete in order
#pragma unroll
  for (int u = 0; u < KU; ++u)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      bf16x8_t hi, lo;
      if constexpr (PRE) {
        hi = bf8(f.b[u][nt][0][0]);
        lo = bf8(f.b[u][nt][0][1]);
      } else {
        sum_split<NP>(f.b[u][nt], hi, lo);
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const bf16x8_t a = bf8(tile[(16 * rt + m) * S::PITCH + 4 * u + g]);
        acc[rt][nt] = mfma16(a, hi, acc[rt][nt]);
        acc[rt][nt] = mfma16(a, lo, acc[rt][nt]);
      }
    }
  __builtin_amdgcn_wave_barrier();
}

// acc[rt][nt] += weight tile rt . token tile nt over the k steps [ks0, ks1) (uniform).
// Two register sets alternate: the loads of the next KU steps are issued before the
// current ones are multiplied; loads past ks1 are out of range and read nothing.  A
// pair always multiplies both halves (a group past ks1 adds zeros) and the exit test
// closes the pair, so no load sits on a conditional path: with an exit test between
// the halves the compiler moved the loads next to their use and waited on them there.
template <int RT, int NT, int KU, int NP, bool PRE = false, class W = WBf16>
__device__ __forceinline__ void stream_rows(const Buf& wb, int C, const int* roff, uint4* tile, const Buf& tb,
                                            uint32_t part_bytes, int tn, int ks0, int ks1, f32x4_t (&acc)[RT][NT]) {
  if (ks0 >= ks1) return;
  Frags<RT, NT, KU, NP, W> f0, f1;
  load_frags<RT, NT, KU, NP, PRE, W>(f0, wb, C, roff, tb, part_bytes, tn, ks0, ks1);
  if (ks0 + KU >= ks1) {  // a single group
    mma_frags<RT, NT, KU, NP, PRE, W>(f0, tile, acc);
    return;
  }
  for (int ks = ks0;; ks += 2 * KU) {
    load_frags<RT, NT, KU, NP, PRE, W>(f1, wb, C, roff, tb, part_bytes, tn, ks + KU, ks1);
    issue_barrier();
    mma_frags<RT, NT, KU, NP, PRE, W>(f0, tile, acc);
    load_frags<RT, NT, KU, NP, PRE, W>(f0, wb, C, roff, tb, part_bytes, tn, ks + 2 * KU, ks1);
    issue_barrier();
    mma_frags<RT, NT, KU, NP, PRE, W>(f1, tile, acc);
    if (ks + 2 * KU >= ks1) break;
  }
}

// The token side of a product with rows of C chunks: fp32 rows of x, or (pre) the
// planes written by k_split_tokens for ntt token tiles.
struct TokSrc {
  Buf b;
  uint32_t part;
  int tn;
};
__device__ __forceinline__ TokSrc token_source(bool pre, const float* x, const uint4* xs, int C, int T, int ntt) {
  if (pre) {
    const uint32_t plane = 16u * (uint32_t)((C + 3) / 4) * (uint32_t)ntt * (uint32_t)kWave;
    return TokSrc{make_buf(xs, 2 * plane), plane, ntt};
  }
  return TokSrc{make_buf(x, 32u * (uint32_t)T * (uint32_t)C), 0u, T};
}

// ------------------------------------------------------------------ token pre-split
// For batches of more than one token tile every gate workgroup multiplies all tokens
// against its rows.  Read as fp32 rows, a token load instruction touches 16 rows (one per
// token of the tile) and half of each cache line it uses, and every workgroup splits
// every value again.  This kernel writes the split once, in fragment order: entry
// ((ks ntt + nt) 64 + lane) of the hi plane holds the bf16 hi parts of tokens
// 16 nt + (lane & 15), elements 32 ks + 8 (lane >> 4) .. + 7, the lo plane (nks ntt 64
// entries later) their lo parts; zero past the batch and past d.
__global__ __launch_bounds__(kBlock) void k_split_tokens(const float* __restrict__ x, int C, int T, int nks, int ntt,
                                                         uint4* __restrict__ xs) {
  const int n = nks * ntt * kWave, i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const int lane = i % kWave, fr = i / kWave, nt = fr % ntt, ks = fr / ntt;
  const int tok = 16 * nt + (lane & 15), c = 4 * ks + (lane >> 4);
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (tok < T && c < C) {
    const float4* p = reinterpret_cast<const float4*>(x + 8 * ((size_t)tok * C + c));
    const float4 a = p[0], b = p[1];
    v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
  }
  bf16x8_t hi, lo;
  split8(v, hi, lo);
  xs[i] = __builtin_bit_cast(uint4, hi);
  xs[n + i] = __builtin_bit_cast(uint4, lo);
}

// ------------------------------------------------------------------ LoPA z = A x
// Workgroup b: 16-row tile of A over one half (kZParts) of the d range, each of its waves a
// sixteenth of that half, for NT token tiles; with pre-split tokens each group of NT token
// tiles has workgroups of its own (at 64 tokens, r = 512: 256 workgroups instead of 64 that
// each read every token's fragments).  The waves' sums are added in LDS (fixed order) and
// stored as partial copy `part` of z: zp[part][tc][r]; the gate kernel adds the two copies.
constexpr int kZWaves = 16;
constexpr int kZParts = 2;

template <int NT, bool PRE, class W>
__global__ __launch_bounds__(kZWaves * kWave) void k_lopa_z_mfma(const float* __restrict__ x,
                                                                 const uint4* __restrict__ xs, int ntt,
                                                                 const uint4* __restrict__ A, int C, int T, int r,
                                                                 int tc, float* __restrict__ zp, GWork gw,
                                                                 const float* __restrict__ s_a) {
  if (g_precompute(gw)) return;
  __shared__ f32x4_t s_part[kZWaves][NT][kWave];
  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  // blockIdx.x = (tile kZParts + part) ngrp + tg: tg the group of NT token tiles
  const int ngrp = PRE ? ntt / NT : 1;
  const int tg = (int)blockIdx.x % ngrp, tp = (int)blockIdx.x / ngrp;
  const int tile = tp / kZParts, part = tp % kZParts;
  constexpr int KU = NT == 1 ? 4 : NT == 2 ? 2 : 1;
  using S = WStage<1, KU, W>;
  __shared__ uint4 s_stage[kZWaves][S::WORDS];
  int roff[S::NI];
  stage_rows<1, KU, W>(roff, C, [&](int br) { return tile * 16 + br < r ? tile * 16 + br : -1; });
  const Buf ab = make_buf(A, 16u * (uint32_t)r * (uint32_t)(C / S::R8));
  TokSrc tok = token_source(PRE, x, xs, C, T, ntt);
  if constexpr (PRE) {  // the group's first token tile at entry 0 of each k step's row of tiles
    const uint32_t skip = 16u * (uint32_t)(tg * NT * kWave);
    tok.b = make_buf(xs + (size_t)tg * NT * kWave, 2 * tok.part - skip);
  }
  f32x4_t acc[1][NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[0][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  int ks0, ks1;
  kpart(C, part * kZWaves + wave, kZParts * kZWaves, &ks0, &ks1);
  stream_rows<1, NT, KU, 1, PRE, W>(ab, C, roff, s_stage[wave], tok.b, tok.part, tok.tn, ks0, ks1, acc);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) s_part[wave][nt][lane] = acc[0][nt];
  __syncthreads();
  // thread o: local token o / 16 of the group, row tile * 16 + o % 16 (16 consecutive floats
  // of z a token); that value sits in lane 16 (kk / 4) + tl % 16, element kk % 4, of the
  // group's token tile tl / 16
  const float* sp = reinterpret_cast<const float*>(s_part);
  const int tok0 = 16 * NT * tg;
  for (int o = threadIdx.x; o < 16 * NT * 16; o += kZWaves * kWave) {
    const int tl = o >> 4, kk = o & 15, tok = tok0 + tl;
    const int k = tile * 16 + kk;
    if (k >= r || tok >= T) continue;
    const int nt = tl >> 4, src = ((16 * (kk >> 2) + (tl & 15)) << 2) + (kk & 3);
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kZWaves; ++w) s += sp[(w * NT + nt) * kWave * 4 + src];
    if constexpr (is_quant<W>()) s *= s_a[k];  // the row's scale
    zp[((size_t)part * tc + tok) * r + k] = s;
  }
}

// ------------------------------------------------------------------ gate + union + W_up
// Segments of at most 64 neurons, each workgroup taking every gridDim.x-th one.  Wave w
// multiplies the segment's four row tiles over k part w; the parts are added in LDS,
// wave w owning tile w.  A neuron joins the union if any token activates it (h > t;
// NaN compares false); one ballot orders the union ascending.  The W_up dots of the
// union rows use the same split, and zval = act * v goes to the fragment buffer of the
// down kernel: per fragment group (segment, entries 32 gi .. 32 gi + 31) and token tile
// a plane of 64 hi entries, then one of 64 lo entries; entry m + 16 g holds, for token
// 16 nt + m, the bf16 parts of entries 4g .. 4g + 3 then 16 + 4g .. 16 + 4g + 3 of the
// group.  A used group is written whole (zero past the union), an unused one is never
// read.
// LOPA: the gate rows are B [d_ff][r] against z = zp[0] + zp[1]; otherwise W_gate x.
// KU / KUU: k steps per load group of the gate rows / the W_up rows.
// FORM (a FormKind): the paper's full form (`form`): the activation value, SiLU on the
// W_up output and, with kFormLoPA, the fixed term G added to the gate before the union.
template <class W, bool LOPA, bool DENSE, int NT, int KU, int KUU, int FORM>
__device__ __forceinline__ void gate_up_body(const float* __restrict__ x, const float* __restrict__ zp,
                                             const uint4* __restrict__ gate_w, int Cg, const uint4* __restrict__ w_up,
                                             int Cu, int T, int d, int d_ff, int nseg, float t, int slots, int tc,
                                             int32_t* __restrict__ meta, int32_t* __restrict__ seg_count,
                                             int32_t* __restrict__ seg_idx, float* __restrict__ seg_act,
                                             uint4* __restrict__ zf, float* __restrict__ y,
                                             const uint4* __restrict__ xs, int ntt, Form form,
                                             const float* __restrict__ gx, const float* __restrict__ s_g,
                                             const float* __restrict__ s_up, const float* __restrict__ s_down) {
  constexpr bool Q = is_quant<W>();
  constexpr int R8 = W::EPC / 8;
  constexpr bool FULL = FORM != kFormDefault, HAS_G = FORM == kFormLoPA;
  constexpr bool PRE = NT > 1;  // tokens pre-split by k_split_tokens
  // the W_up rows of a union of at most two row tiles go as two tiles with twice the k
  // steps a group (one token tile only: the register budget of wider ones is spent)
  constexpr bool NARROW = NT == 1;
  constexpr int STAGE_A = WStage<kTiles, (KU > KUU ? KU : KUU)>::WORDS, STAGE_B = WStage<2, 2 * KUU>::WORDS;
  constexpr int STAGE = NARROW && STAGE_B > STAGE_A ? STAGE_B : STAGE_A;
  __shared__ uint4 s_stage[kParts][STAGE];
  __shared__ f32x4_t s_red[kParts][kTiles][NT][kWave];
  __shared__ float s_act[kSegRowsB][16 * NT];
  __shared__ uint32_t s_mask[kTiles];
  __shared__ int s_list[kSegRowsB];
  __shared__ int s_cnt;

  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  const int m = lane & 15, g = lane >> 4;
  clear_output(y, T * d, meta, nseg);
  const TokSrc tok = token_source(PRE, x, xs, Cu, T, ntt);
  const Buf ub = make_buf(w_up, 16u * (uint32_t)d_ff * (uint32_t)(Cu / R8));

  // segments blockIdx.x, blockIdx.x + gridDim.x, ... (the host makes the counts equal)
  const Split segs(d_ff, nseg);
  for (int seg = blockIdx.x; seg < nseg; seg += gridDim.x) {
    if (seg != (int)blockIdx.x) __syncthreads();  // the previous segment's LDS reads are done
    const int row0 = segs.start(seg);
    const int nrows = segs.start(seg + 1) - row0;  // <= kSegRowsB, guaranteed by the host

    f32x4_t acc[kTiles][NT];
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[rt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    {
      int roff[WStage<kTiles, KU, W>::NI];
      stage_rows<kTiles, KU, W>(roff, Cg, [&](int br) { return br < nrows ? row0 + br : -1; });
      int ks0, ks1;
      kpart(Cg, wave, kParts, &ks0, &ks1);
      const Buf gb = make_buf(gate_w, 16u * (uint32_t)d_ff * (uint32_t)(Cg / R8));
      if constexpr (LOPA) {
        const uint32_t part = 32u * (uint32_t)tc * (uint32_t)Cg;
        stream_rows<kTiles, NT, KU, 2, false, W>(gb, Cg, roff, s_stage[wave], make_buf(zp, 2 * part), part, T, ks0,
                                                 ks1, acc);
      } else {
        stream_rows<kTiles, NT, KU, 1, PRE, W>(gb, Cg, roff, s_stage[wave], tok.b, tok.part, tok.tn, ks0, ks1, acc);
      }
    }
    // LoPA's fixed term (G x) of the rows and tokens this lane thresholds, written by the z
    // kernel's extra workgroups: loaded after the gate stream (no registers held across
    // it), so that the wait falls after the LDS reduction
    uint32_t gxb[HAS_G ? NT : 1][4] = {};
    if constexpr (HAS_G) {
      const Buf xb = make_buf(gx, 4u * (uint32_t)tc * (uint32_t)d_ff);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * nt + m, rl = 16 * wave + 4 * g + i;
          gxb[nt][i] = ldb32(xb, tok < T && rl < nrows ? 4u * ((uint32_t)tok * (uint32_t)d_ff + (uint32_t)(row0 + rl))
                                                        : kOOB);
        }
    }
    // quantized: the row scales of the rows this lane thresholds (likewise after the stream)
    uint32_t sgb[Q ? 4 : 1] = {};
    if constexpr (Q) {
      const Buf qb = make_buf(s_g, 4u * (uint32_t)d_ff);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = 16 * wave + 4 * g + i;
        sgb[i] = ldb32(qb, rl < nrows ? 4u * (uint32_t)(row0 + rl) : kOOB);
      }
    }
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) s_red[wave][rt][nt][lane] = acc[rt][nt];
    __syncthreads();
    {
      // lane holds h of rows 16 wave + 4g + i (i < 4) for tokens 16 nt + m
      f32x4_t h[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        h[nt] = ((s_red[0][wave][nt][lane] + s_red[1][wave][nt][lane]) + s_red[2][wave][nt][lane]) +
                s_red[3][wave][nt][lane];
      uint32_t mask = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = 16 * wave + 4 * g + i;
        bool any = false;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int tok = 16 * nt + m;
          float hv = h[nt][i];
          if constexpr (Q) hv *= __builtin_bit_cast(float, sgb[i]);
          if constexpr (HAS_G) hv += __builtin_bit_cast(float, gxb[nt][i]);  // h += G x
          const bool on = tok < T && hv > t;
          if (tok < T && rl < nrows) s_act[rl][tok] = on ? (FULL ? gate_value(form.act, hv - t) : hv - t) : 0.f;
          any |= on;
        }
        const uint64_t b = __ballot(any && rl < nrows);
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
          if ((b >> (16 * gg)) & 0xffffull) mask |= 1u << (4 * gg + i);
      }
      if (lane == 0) s_mask[wave] = mask;
    }
    __syncthreads();
    if (wave == 0) {
      const uint64_t on = (uint64_t)s_mask[0] | ((uint64_t)s_mask[1] << 16) | ((uint64_t)s_mask[2] << 32) |
                          ((uint64_t)s_mask[3] << 48);
      const bool sel = lane < nrows && (DENSE || ((on >> lane) & 1ull));
      const uint64_t b = __ballot(sel);
      const int rank = rank_in_mask(b);
      if (sel) {
        s_list[rank] = lane;
        seg_idx[row0 + rank] = row0 + lane;
      }
      if (lane == 0) {
        s_cnt = __popcll(b);
        seg_count[seg] = __popcll(b);
      }
    }
    __syncthreads();
    const int cnt = uniform(s_cnt);
    for (int o = threadIdx.x; o < cnt * T; o += kBlock) {
      const int tok = o / cnt, e = o - tok * cnt;
      seg_act[(size_t)tok * slots + row0 + e] = s_act[s_list[e]][tok];
    }

    // W_up dots of the union rows: tiles of 16 entries
    const int nut = (cnt + 15) / 16;
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[rt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (nut > 0) {
      int ks0, ks1;
      kpart(Cu, wave, kParts, &ks0, &ks1);
      auto up_row = [&](int e) { return e < cnt ? row0 + s_list[e] : -1; };
      auto full = [&] {
        int roff[WStage<kTiles, KUU, W>::NI];
        stage_rows<kTiles, KUU, W>(roff, Cu, up_row);
        stream_rows<kTiles, NT, KUU, 1, PRE, W>(ub, Cu, roff, s_stage[wave], tok.b, tok.part, tok.tn, ks0, ks1, acc);
      };
      if constexpr (NARROW) {
        if (nut <= 2) {
          int roff[WStage<2, 2 * KUU, W>::NI];
          stage_rows<2, 2 * KUU, W>(roff, Cu, up_row);
          stream_rows<2, NT, 2 * KUU, 1, false, W>(ub, Cu, roff, s_stage[wave], tok.b, tok.part, tok.tn, ks0, ks1,
                                                   reinterpret_cast<f32x4_t(&)[2][NT]>(acc));
        } else {
          full();
        }
      } else {
        full();
      }
    }
#pragma unroll
    for (int rt = 0; rt < kTiles; ++rt)
      if (rt < nut)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) s_red[wave][rt][nt][lane] = acc[rt][nt];
    __syncthreads();

    // wave w: union entries 16 w .. 16 w + 15 = half (w & 1) of fragment group w >> 1
    const int gi = wave >> 1, half = wave & 1;
    // quantized: the W_up scale of each entry's row, and its W_down scale folded into zval
    float sue[4] = {1.f, 1.f, 1.f, 1.f}, sde[4] = {1.f, 1.f, 1.f, 1.f};
    if constexpr (Q) {
      const Buf ubs = make_buf(s_up, 4u * (uint32_t)d_ff), dbs = make_buf(s_down, 4u * (uint32_t)d_ff);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = 16 * wave + 4 * g + i;
        const uint32_t off = e < cnt ? 4u * (uint32_t)(row0 + s_list[e < cnt ? e : 0]) : kOOB;
        sue[i] = __builtin_bit_cast(float, ldb32(ubs, off));
        sde[i] = __builtin_bit_cast(float, ldb32(dbs, off));
      }
    }
    if (32 * gi < cnt) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int tok = 16 * nt + m;
        f32x4_t v = {0.f, 0.f, 0.f, 0.f};
        if (wave < nut)
          v = ((s_red[0][wave][nt][lane] + s_red[1][wave][nt][lane]) + s_red[2][wave][nt][lane]) +
              s_red[3][wave][nt][lane];
        if (tok < T) {
          uint32_t hw[2] = {0u, 0u}, lw[2] = {0u, 0u};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int e = 16 * wave + 4 * g + i;
            const float vu = Q ? v[i] * sue[i] : v[i];
            float zz = e < cnt ? s_act[s_list[e]][tok] * (FULL ? up_value(form.silu_up, vu) : vu) : 0.f;
            if constexpr (Q) zz *= sde[i];
            const __bf16 hb = (__bf16)zz;
            const __bf16 lb = (__bf16)(zz - (float)hb);
            hw[i >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, hb) << (16 * (i & 1));
            lw[i >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, lb) << (16 * (i & 1));
          }
          // hi plane entry of lane m + 16 g, then the lo plane 64 entries on
          uint4* frag = zf + ((((size_t)seg * 2 + gi) * ntt + nt) * 2) * kWave + m + 16 * g;
          reinterpret_cast<uint2*>(frag)[half] = make_uint2(hw[0], hw[1]);
          reinterpret_cast<uint2*>(frag + kWave)[half] = make_uint2(lw[0], lw[1]);
        }
      }
    }
  }
}

#define FFN_GATE_UP_PARAMS                                                                                         \
  const float *__restrict__ x, const float *__restrict__ zp, const uint4 *__restrict__ gate_w, int Cg,             \
      const uint4 *__restrict__ w_up, int Cu, int T, int d, int d_ff, int nseg, float t, int slots, int tc,       \
      int32_t *__restrict__ meta, int32_t *__restrict__ seg_count, int32_t *__restrict__ seg_idx,                  \
      float *__restrict__ seg_act, uint4 *__restrict__ zf, float *__restrict__ y, const uint4 *__restrict__ xs,  \
      int ntt, Form form, const float *__restrict__ gx, const float *__restrict__ s_g,                            \
      const float *__restrict__ s_up, const float *__restrict__ s_down
#define FFN_GATE_UP_ARGS                                                                                            \
  x, zp, gate_w, Cg, w_up, Cu, T, d, d_ff, nseg, t, slots, tc, meta, seg_count, seg_idx, seg_act, zf, y, xs, ntt, form, \
      gx, s_g, s_up, s_down

// One workgroup per CU: four k steps a group for one token tile (two for LoPA's short
// gate rows and for wider token tiles; one for LoPA's gate rows with four token tiles,
// whose fragments carry both partial copies of z).
template <class W, bool LOPA, bool DENSE, int NT, int FORM>
__global__ __launch_bounds__(kBlock) void k_gate_up_mfma(FFN_GATE_UP_PARAMS) {
  constexpr int KU = NT == 1 ? (LOPA ? 2 : 4) : (LOPA && NT == 4 ? 1 : 2);
  gate_up_body<W, LOPA, DENSE, NT, KU, NT == 1 ? 4 : 2, FORM>(FFN_GATE_UP_ARGS);
}

// One token tile: two k steps a group, so that two workgroups fit a CU (at most 256
// registers a lane); one workgroup's phase changes (LDS reductions, union) then overlap the
// other's streaming.  LoPA's gate rows keep two k steps a group as in k_gate_up_mfma.
template <class W, bool LOPA, bool DENSE, int FORM>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(2))) void k_gate_up_mfma2(
    FFN_GATE_UP_PARAMS) {
  gate_up_body<W, LOPA, DENSE, 1, 2, 2, FORM>(FFN_GATE_UP_ARGS);
}
// ------------------------------------------------------------------ batches of 2 .. 4 tokens
// For at most four tokens the gate and the W_up dots run on v_mfma_f32_4x4x4_16b_bf16:
// sixteen independent 4x4x4 products an instruction, in which lane 4b + i holds 4
// consecutive k of row i of block b (A operand), lane 4b + j those of token j (B operand),
// and element i of lane 4b + j receives D[b][i][j].  One load instruction of a quad (four
// rows) gives lane 4b + i the 16-byte chunk b of 16 consecutive chunks of row i: 256
// contiguous bytes a row, already in the A layout (its 8 bf16, or 16 / 32 codes converted
// to bf16, feed 2 / 4 / 8 products), so rows need no reshaping through LDS and a quad of
// union rows is any four rows.  The 16 blocks hold disjoint k ranges of the same 4 x 4
// product and are summed once the quad is done.  The tokens (x, and LoPA's z: the sum of the
// z kernel's two partial copies) sit in LDS, split once per workgroup into bf16 hi + lo in
// the order the lanes read them, so the streams load nothing but weights.  Eight waves a workgroup with four loads in flight each (32 KB a CU) measured
// fastest: at 8B int8 / int4 and four tokens the gate kernel took 22.6 / 22.5 us, against
// 26.1 / 25.9 us with sixteen waves and eight loads, 30.2 / 28.2 us with sixteen and twelve,
// and 33.3 / 28.2 us with four waves and four loads.  Tokens past the batch are zeros (a batch
// of 2 or 3 tokens leaves lanes idle).
// Against the 16x16x32 kernel at four tokens on the 8B shape: standard gating with int8 /
// int4 rows 42.1 / 41.9 -> 32.6 / 32.1 us a call; LoPA (r = 512) with bf16 / int8 / int4 rows
// 38.4 / 34.7 / 34.3 -> 37.7 / 31.8 / 31.5 us.
constexpr int kQ4Waves = 8;       // waves a workgroup (one workgroup a CU: two a SIMD)
constexpr int kQ4Threads = kQ4Waves * kWave;
constexpr int kQ4Depth = 4;       // weight loads in flight a wave
constexpr int kQ4MaxX = 4096;     // elements a token: x (d padded to a whole step) ...
constexpr int kQ4MaxZ = 1024;     // ... and LoPA's z (r padded likewise)
constexpr int kQ4Quads = kSegRowsB / 4;

__device__ __forceinline__ short4_t half4(const uint4& v, int h) {
  return __builtin_bit_cast(short4_t, h ? make_uint2(v.z, v.w) : make_uint2(v.x, v.y));
}
__device__ __forceinline__ f32x4_t mfma4(short4_t a, short4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a, b, c, 0, 0, 0);
}

// One step of a quad: the weight chunk v (8 elements a 16-byte group J) against the token
// fragment at t: t[f kWave], f < FW / 2 the hi parts, then as many lo parts.  Four accumulators take the
// hi and lo products of the two k halves of each group, so that no product waits on the
// one before it.
template <class W>
__device__ __forceinline__ void q4_mma(const uint4& v, const uint4* __restrict__ t, f32x4_t (&acc)[4]) {
  constexpr int G8 = W::EPC / 8, FW = W::EPC / 4;
  auto one = [&](const uint4& w, const uint4& th, const uint4& tl) {
    acc[0] = mfma4(half4(w, 0), half4(th, 0), acc[0]);
    acc[1] = mfma4(half4(w, 0), half4(tl, 0), acc[1]);
    acc[2] = mfma4(half4(w, 1), half4(th, 1), acc[2]);
    acc[3] = mfma4(half4(w, 1), half4(tl, 1), acc[3]);
  };
  one(bf16_chunk<W, 0>(v), t[0], t[(FW / 2) * kWave]);
  if constexpr (G8 > 1) one(bf16_chunk<W, 1>(v), t[kWave], t[(FW / 2 + 1) * kWave]);
  if constexpr (G8 > 2) {
    one(bf16_chunk<W, 2>(v), t[2 * kWave], t[(FW / 2 + 2) * kWave]);
    one(bf16_chunk<W, 3>(v), t[3 * kWave], t[(FW / 2 + 3) * kWave]);
  }
}

// Items [i0, i1) of a quad stream: item it is step it % ns of quad it / ns; a step is 16
// chunks of a row (C chunks a row, ns = ceil(C / 16) steps).  row_of(q) is this lane's row
// of quad q (row lane & 3 of the quad), or -1.  The weights of item it + kQ4Depth are
// requested when item it has been multiplied; items past i1 load nothing.  deposit(q, s)
// receives the quad's 4 x 4 sums in lanes 0..3 (lane j: s[i] = row i . token j) when the
// stream leaves quad q.  stage() runs once the first loads are out, in every thread.
template <class W, class RowOf, class Stage, class Deposit>
__device__ __forceinline__ void q4_stream(const Buf& wb, int C, int ns, int i0, int i1,
                                          const uint4* __restrict__ tok, RowOf row_of, Stage stage,
                                          Deposit deposit) {
  constexpr int D = kQ4Depth, FW = W::EPC / 4;
  const int lane = lane_id(), b = lane >> 2;
  uint4 wv[D];
  int lq = i0 / ns, ls = i0 - lq * ns;
  int lrow = row_of(lq);
  auto issue = [&](int u, bool live) {
    const int ch = 16 * ls + b;
    wv[u] = ldb_nt(wb, live && lrow >= 0 && ch < C ? 16u * ((uint32_t)lrow * (uint32_t)C + (uint32_t)ch) : kOOB);
    if (live && ++ls == ns) {
      ls = 0;
      lrow = row_of(++lq);
    }
  };
  int cq = i0 / ns, cs = i0 - cq * ns;
#pragma unroll
  for (int u = 0; u < D; ++u) issue(u, i0 + u < i1);
  stage();
  f32x4_t acc[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) acc[a] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto flush = [&] {
    f32x4_t s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
#pragma unroll
    for (int o = 4; o < kWave; o <<= 1)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[i] += __shfl_xor(s[i], o);
    deposit(cq, s);
#pragma unroll
    for (int a = 0; a < 4; ++a) acc[a] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  };
  for (int it = i0; it < i1; it += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      if (it + u < i1) {
        q4_mma<W>(wv[u], tok + (size_t)cs * FW * kWave + lane, acc);
        if (++cs == ns) {
          flush();
          cs = 0;
          ++cq;
        }
      }
      issue(u, it + u + D < i1);
    }
  }
  if (cs != 0) flush();  // a quad cut by the end of the range
}

// Tokens into LDS: elements [0, K) of rows j < T of src (row stride `stride` floats; with
// copies = 2 the sum of two partial copies `part` floats apart), split into bf16 hi + lo, for lane 4 ((k / EPC) % 16) + j of step k / (16 EPC): part f of a lane's fragment
// (f < FW / 2 hi, then lo) at uint4 (step FW + f) kWave + lane, so that the lanes of a
// wave read 16 consecutive bytes each.  Zeros up to Kp (a whole number of steps) and for
// rows j >= T.  A region of Kp elements takes Kp uint4.  UMAX: the most 8-element units
// a thread takes (4 Kp / 8 <= UMAX kQ4Threads).  The loads are issued by q4_load_tokens and
// the values stored by q4_store_tokens, so that other loads can go out in between.
template <class W, int UMAX>
__device__ __forceinline__ void q4_load_tokens(const float* __restrict__ src, int T, int K, int Kp, int stride,
                                               float4 (&v)[UMAX][2], int copies = 1, uint32_t part = 0) {
  const Buf sb = make_buf(src, 4u * (copies == 2 ? 2u * part : (uint32_t)T * (uint32_t)stride));
  const int nu = 4 * (Kp / 8);
#pragma unroll
  for (int u = 0; u < UMAX; ++u) {
    const int unit = threadIdx.x + u * kQ4Threads, j = unit % 4, k = 8 * (unit / 4);
    const bool ok = unit < nu && j < T && k < K;
    const uint32_t off = ok ? 4u * ((uint32_t)j * (uint32_t)stride + (uint32_t)k) : kOOB;
    float4 a = __builtin_bit_cast(float4, ldb(sb, off)), c = __builtin_bit_cast(float4, ldb(sb, off + 16));
    if (copies == 2) {
      const float4 a2 = __builtin_bit_cast(float4, ldb(sb, ok ? off + 4u * part : kOOB));
      const float4 c2 = __builtin_bit_cast(float4, ldb(sb, ok ? off + 4u * part + 16 : kOOB));
      a = make_float4(a.x + a2.x, a.y + a2.y, a.z + a2.z, a.w + a2.w);
      c = make_float4(c.x + c2.x, c.y + c2.y, c.z + c2.z, c.w + c2.w);
    }
    v[u][0] = a;
    v[u][1] = c;
  }
}
template <class W, int UMAX>
__device__ __forceinline__ void q4_store_tokens(const float4 (&v)[UMAX][2], int Kp, uint4* __restrict__ tok) {
  constexpr int EPC = W::EPC, FW = EPC / 4;
  const int nu = 4 * (Kp / 8);
#pragma unroll
  for (int u = 0; u < UMAX; ++u) {
    const int unit = threadIdx.x + u * kQ4Threads, j = unit % 4, k = 8 * (unit / 4);
    if (unit < nu) {
      const float f[8] = {v[u][0].x, v[u][0].y, v[u][0].z, v[u][0].w, v[u][1].x, v[u][1].y, v[u][1].z, v[u][1].w};
      bf16x8_t hi, lo;
      split8(f, hi, lo);
      const int step = k / (16 * EPC), bb = (k / EPC) % 16, grp = (k % EPC) / 8;
      uint4* p = tok + (size_t)step * FW * kWave + 4 * bb + j;
      p[grp * kWave] = __builtin_bit_cast(uint4, hi);
      p[(FW / 2 + grp) * kWave] = __builtin_bit_cast(uint4, lo);
    }
  }
}

// Gate, union and W_up dots of one segment for batches of at most four tokens (the same
// outputs as gate_up_body with one token tile).  Every wave takes an equal share of the
// segment's (quad, step) items, so a quad may be split between waves: each wave leaves its
// partial sums in its own LDS slots and the slots are added in a fixed order.
template <class W, bool LOPA, bool DENSE, int FORM>
__global__ __launch_bounds__(kQ4Threads) void k_gate_up_q4(FFN_GATE_UP_PARAMS) {
  constexpr int EPC = W::EPC, STEP = 16 * EPC;
  constexpr bool Q = is_quant<W>();
  constexpr bool FULL = FORM != kFormDefault, HAS_G = FORM == kFormLoPA;
  constexpr int UX = 4 * kQ4MaxX / 8 / kQ4Threads, UZ = LOPA ? (4 * kQ4MaxZ / 8 + kQ4Threads - 1) / kQ4Threads : 1;
  __shared__ uint4 s_tok[kQ4MaxX + (LOPA ? kQ4MaxZ : 0)];
  // partial sums [wave][quad][token] (element i: row i of the quad) of the gate and W_up
  __shared__ f32x4_t s_pg[kQ4Waves][kQ4Quads][4], s_pu[kQ4Waves][kQ4Quads][4];
  __shared__ float s_act[kSegRowsB][4];
  __shared__ int s_list[kSegRowsB];
  __shared__ int s_cnt;

  const int lane = lane_id(), wave = uniform(threadIdx.x / kWave);
  for (int j = blockIdx.x * kQ4Threads + threadIdx.x; j < T * d; j += gridDim.x * kQ4Threads) y[j] = 0.f;
  if (blockIdx.x == 0 && threadIdx.x == 0) meta[0] = nseg;
  const int Cu_ = Cu / (EPC / 8), Cg_ = Cg / (EPC / 8);
  const int nsu = (Cu_ + 15) / 16, Kpx = nsu * STEP, nsg = (Cg_ + 15) / 16, Kpz = LOPA ? nsg * STEP : 0;
  uint4* const tok_g = s_tok + (LOPA ? Kpx : 0);
  const Buf gb = make_buf(gate_w, 16u * (uint32_t)d_ff * (uint32_t)Cg_);
  const Buf ub = make_buf(w_up, 16u * (uint32_t)d_ff * (uint32_t)Cu_);
  auto deposit_g = [&](int q, const f32x4_t& s) {
    if (lane < 4) s_pg[wave][q][lane] = s;
  };
  auto deposit_u = [&](int q, const f32x4_t& s) {
    if (lane < 4) s_pu[wave][q][lane] = s;
  };

  const Split segs(d_ff, nseg);
  bool staged = false;
  for (int seg = blockIdx.x; seg < nseg; seg += gridDim.x) {
    __syncthreads();  // the previous segment's LDS reads are done
    const int row0 = segs.start(seg);
    const int nrows = segs.start(seg + 1) - row0;  // <= kSegRowsB, guaranteed by the host
    for (int o = threadIdx.x; o < kQ4Waves * kQ4Quads * 4; o += kQ4Threads) {
      (&s_pg[0][0][0])[o] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      (&s_pu[0][0][0])[o] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    {
      const int n = ((nrows + 3) / 4) * nsg;
      const int i0 = (int)((int64_t)n * wave / kQ4Waves), i1 = (int)((int64_t)n * (wave + 1) / kQ4Waves);
      auto row_of = [&](int q) {
        const int rl = 4 * q + (lane & 3);
        return rl < nrows ? row0 + rl : -1;
      };
      auto stage = [&] {
        if (staged) return;
        staged = true;
        float4 vx[UX][2];
        q4_load_tokens<W, UX>(x, T, d, Kpx, d, vx);
        float4 vz[UZ][2];
        if constexpr (LOPA) q4_load_tokens<W, UZ>(zp, T, Cg * 8, Kpz, Cg * 8, vz, 2, (uint32_t)tc * (uint32_t)Cg * 8u);
        q4_store_tokens<W, UX>(vx, Kpx, s_tok);
        if constexpr (LOPA) q4_store_tokens<W, UZ>(vz, Kpz, tok_g);
        __syncthreads();
      };
      if (i0 < i1)
        q4_stream<W>(gb, Cg_, nsg, i0, i1, tok_g, row_of, stage, deposit_g);
      else
        stage();
    }
    // the row scale of the row this lane of wave 0 thresholds
    float sg = 1.f, gxv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (Q)
      if (wave == 0)
        sg = __int_as_float(ldb32(make_buf(s_g, 4u * (uint32_t)d_ff), lane < nrows ? 4u * (uint32_t)(row0 + lane) : kOOB));
    if constexpr (HAS_G)
      if (wave == 0) {
        const Buf xb = make_buf(gx, 4u * (uint32_t)tc * (uint32_t)d_ff);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          gxv[j] = __int_as_float(
              ldb32(xb, j < T && lane < nrows ? 4u * ((uint32_t)j * (uint32_t)d_ff + (uint32_t)(row0 + lane)) : kOOB));
      }
    __syncthreads();
    if (wave == 0) {
      // lane: row `lane` of the segment
      const int q = lane >> 2, i = lane & 3;
      bool any = false;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float hv = 0.f;
#pragma unroll
        for (int w = 0; w < kQ4Waves; ++w) hv += s_pg[w][q][j][i];
        if constexpr (Q) hv *= sg;
        if constexpr (HAS_G) hv += gxv[j];
        const bool on = j < T && hv > t;
        if (lane < nrows) s_act[lane][j] = on ? (FULL ? gate_value(form.act, hv - t) : hv - t) : 0.f;
        any |= on;
      }
      const bool sel = lane < nrows && (DENSE || any);
      const uint64_t bm = __ballot(sel);
      const int rank = rank_in_mask(bm);
      if (sel) {
        s_list[rank] = lane;
        seg_idx[row0 + rank] = row0 + lane;
      }
      if (lane == 0) {
        s_cnt = __popcll(bm);
        seg_count[seg] = __popcll(bm);
      }
    }
    __syncthreads();
    const int cnt = uniform(s_cnt);
    for (int o = threadIdx.x; o < cnt * T; o += kQ4Threads) {
      const int tk = o / cnt, e = o - tk * cnt;
      seg_act[(size_t)tk * slots + row0 + e] = s_act[s_list[e]][tk];
    }
    {
      const int n = ((cnt + 3) / 4) * nsu;
      const int i0 = (int)((int64_t)n * wave / kQ4Waves), i1 = (int)((int64_t)n * (wave + 1) / kQ4Waves);
      auto row_of = [&](int q) {
        const int e = 4 * q + (lane & 3);
        return e < cnt ? row0 + s_list[e] : -1;
      };
      if (i0 < i1) q4_stream<W>(ub, Cu_, nsu, i0, i1, s_tok, row_of, [] {}, deposit_u);
    }
    __syncthreads();

    // wave w: union entries 16 w .. 16 w + 15 = half (w & 1) of fragment group w >> 1;
    // lane m + 16 g: token m, entries 16 w + 4 g + i
    const int m = lane & 15, g = lane >> 4;
    const int gi = wave >> 1, half = wave & 1;
    float sue[4] = {1.f, 1.f, 1.f, 1.f}, sde[4] = {1.f, 1.f, 1.f, 1.f};
    if constexpr (Q) {
      const Buf ubs = make_buf(s_up, 4u * (uint32_t)d_ff), dbs = make_buf(s_down, 4u * (uint32_t)d_ff);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = 16 * (wave & 3) + 4 * g + i;
        const uint32_t off = e < cnt ? 4u * (uint32_t)(row0 + s_list[e < cnt ? e : 0]) : kOOB;
        sue[i] = __int_as_float(ldb32(ubs, off));
        sde[i] = __int_as_float(ldb32(dbs, off));
      }
    }
    if (wave < 4 && 32 * gi < cnt && m < T) {
      const int qq = 4 * wave + g;  // the quad of entries 16 w + 4 g ..
      f32x4_t v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kQ4Waves; ++w) v += s_pu[w][qq][m];
      uint32_t hw[2] = {0u, 0u}, lw[2] = {0u, 0u};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = 16 * wave + 4 * g + i;
        const float vu = Q ? v[i] * sue[i] : v[i];
        float zz = e < cnt ? s_act[s_list[e]][m] * (FULL ? up_value(form.silu_up, vu) : vu) : 0.f;
        if constexpr (Q) zz *= sde[i];
        const __bf16 hb = (__bf16)zz;
        const __bf16 lb = (__bf16)(zz - (float)hb);
        hw[i >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, hb) << (16 * (i & 1));
        lw[i >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, lb) << (16 * (i & 1));
      }
      // token tile 0: hi plane entry of lane m + 16 g, then the lo plane 64 entries on
      uint4* frag = zf + (((size_t)seg * 2 + gi) * ntt * 2) * kWave + m + 16 * g;
      reinterpret_cast<uint2*>(frag)[half] = make_uint2(hw[0], hw[1]);
      reinterpret_cast<uint2*>(frag + kWave)[half] = make_uint2(lw[0], lw[1]);
    }
  }
}

#undef FFN_GATE_UP_PARAMS
#undef FFN_GATE_UP_ARGS

// ------------------------------------------------------------------ down projection
// Workgroup b: column group b % S, row chunk b / S (a balanced share of the segments).
// A wave owns DT 32-column tiles (DT = 4 for one token tile, else 2); a column group
// is CW of them, and wave w takes column slot w % CW and every (4 / CW)-th used
// fragment group of the chunk (32 union entries of one segment).  A group's 32 W_down
// rows are read (64 / 4 DT) rows x 64 DT bytes per instruction, streamed past the
// caches, and written to a wave-private LDS tile; transposing LDS reads
// (ds_read_b64_tr_b16) then hand every lane the 8 entries of one column that the
// matrix-core B operand takes.  The chunk's slot indices and a table of its groups are
// staged in LDS once; the loop reads a group's table entry two groups ahead and its slot
// indices one group ahead, so the weight loads of the next group issue without waiting
// on LDS.  The waves' sums meet in LDS, then go to y with one fp32 atomic per token and
// column (y was cleared by the gate kernel).
constexpr int kDnSlots = 4096;  // most slot indices of one row chunk

template <int NT, class W = WBf16>
struct DnCfg {
  static constexpr int DT = NT == 1 ? 4 : 2;  // 32-column tiles per wave
  static constexpr int CW = NT == 4 ? 1 : 2;  // column slots per workgroup
  static constexpr int WCOLS = 32 * DT * CW;  // columns per workgroup
  static constexpr int R8 = W::EPC / 8;       // tile chunks (8 bf16) per loaded chunk
  static constexpr int LPR = 4 * DT / R8;     // lanes per row of a load instruction
  static constexpr int RPI = kWave / LPR;     // rows per load instruction
  static constexpr int NI = 32 / RPI;         // load instructions per group
  // chunks per LDS row: two pad chunks put the 8 rows that a half-wave's transposing
  // reads touch on distinct banks
  static constexpr int PITCH = 4 * DT + 2;
};

template <int NT, class W = WBf16>
struct DnFrags {
  uint4 t[DnCfg<NT, W>::NI];  // W_down chunks as loaded: entry RPI i + lane / LPR, chunk lane % LPR
  uint4 zh[NT], zl[NT];       // zval fragments (hi, lo) of the token tiles
};

// A group's table entry: x = first slot (relative to the chunk's first row) | entries
// << 16, y = the group's index in the zval fragment buffer.  The kDnPad table entries
// past the last group are empty, so every load of such a group reads nothing.
constexpr int kDnPad = 4 * kParts;

template <int NT, class W = WBf16>
struct DnRows {
  int row[DnCfg<NT, W>::NI];  // neuron of the entry this lane loads, -1 for none
  int2 info;
};

// C: loaded chunks per row, ch: this lane's chunk
template <int NT, class W>
__device__ __forceinline__ DnRows<NT, W> dn_rows(int2 info, const int* s_idx, int C, int ch) {
  using K = DnCfg<NT, W>;
  const int lane = lane_id(), base = info.x & 0xFFFF, cnt = info.x >> 16;
  DnRows<NT, W> a;
  a.info = info;
#pragma unroll
  for (int i = 0; i < K::NI; ++i) {
    const int e = K::RPI * i + lane / K::LPR;
    const bool ok = e < cnt && ch < C;
    const int v = s_idx[ok ? base + e : 0];
    a.row[i] = ok ? v : -1;
  }
  return a;
}

template <int NT, class W>
__device__ __forceinline__ void dn_issue(DnFrags<NT, W>& f, const DnRows<NT, W>& a, const Buf& db, const Buf& zb,
                                         int C, int ch, int T, int ntt) {
  using K = DnCfg<NT, W>;
  const int lane = lane_id(), m = lane & 15;
#pragma unroll
  for (int i = 0; i < K::NI; ++i) f.t[i] = ldb_nt(db, a.row[i] >= 0 ? 16u * (uint32_t)(a.row[i] * C + ch) : kOOB);
  const bool has = a.info.x >> 16 > 0;
  const uint32_t zg = (uint32_t)a.info.y * (uint32_t)ntt;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int tok = 16 * nt + m;
    const uint32_t off = (has && tok < T) ? 16u * (((zg + nt) * 2) * kWave + lane) : kOOB;
    f.zh[nt] = ldb(zb, off);
    f.zl[nt] = ldb(zb, off + 16 * kWave);
  }
}

__device__ __forceinline__ uint2 lds_read_tr16(const char* p) {
  const short4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(p));
  return __builtin_bit_cast(uint2, v);
}

// tile: this wave's LDS tile (32 PITCH uint4).  Within each 16-lane group q of the
// transposing read, lane 4a + b addresses 8 bytes (4 columns) of one tile row and lane
// 4b + c receives element c of the chunks of lanes b, 4 + b, 8 + b, 12 + b.  With lane
// 4a + b pointing at entry 4q + a (then 16 + 4q + a), columns 4b .. 4b + 3 of a 16-column
// block, lane n of the group ends with entries 4q .. 4q + 3 (then 16 + 4q ..) of column
// n: the B operand in the entry order of the zval fragments.
template <int NT, class W>
__device__ __forceinline__ void dn_mma(const DnFrags<NT, W>& f, uint4* tile,
                                       f32x4_t (&acc)[DnCfg<NT, W>::DT][2][NT]) {
  using K = DnCfg<NT, W>;
  constexpr int ROWB = 16 * K::PITCH;  // bytes per tile row
  const int lane = lane_id();
#pragma unroll
  for (int i = 0; i < K::NI; ++i)  // quantized rows: the codes as bf16, R8 tile chunks a loaded chunk
    put_bf16_chunks<W>(tile + (K::RPI * i + lane / K::LPR) * K::PITCH + (lane % K::LPR) * K::R8, f.t[i]);
  __builtin_amdgcn_wave_barrier();  // LDS operations of a wave complete in order
  const char* src = reinterpret_cast<const char*>(tile) + (4 * (lane >> 4) + ((lane >> 2) & 3)) * ROWB + 8 * (lane & 3);
#pragma unroll
  for (int ct = 0; ct < K::DT; ++ct)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint2 lo = lds_read_tr16(src + 64 * ct + 32 * h);
      const uint2 hi = lds_read_tr16(src + 16 * ROWB + 64 * ct + 32 * h);
      const bf16x8_t b = bf8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[ct][h][nt] = mfma16(bf8(f.zh[nt]), b, acc[ct][h][nt]);
        acc[ct][h][nt] = mfma16(bf8(f.zl[nt]), b, acc[ct][h][nt]);
      }
    }
  __builtin_amdgcn_wave_barrier();
}

// C: loaded chunks per row of w_down_t (d / W::EPC); the W_down row scales of quantized
// weights are folded into zval by the gate kernel.
template <int NT, class W>
__global__ __launch_bounds__(kBlock) void k_down_mfma(const int32_t* __restrict__ seg_count,
                                                      const int32_t* __restrict__ seg_idx,
                                                      const uint4* __restrict__ zf, int nseg, int d_ff, int R, int tc,
                                                      const uint4* __restrict__ w_down_t, int C, int d, int T,
                                                      float* __restrict__ y) {
  using K = DnCfg<NT, W>;
  constexpr int CW = K::CW, GS = kParts / CW, WCOLS = K::WCOLS;
  const Buf db = make_buf(w_down_t, 16u * (uint32_t)d_ff * (uint32_t)C);
  const int ntt = (tc + 15) / 16;
  const Buf zb = make_buf(zf, 4096u * (uint32_t)nseg * (uint32_t)ntt);
  // LDS: the waves' tiles and the chunk's slot indices during the loop; afterwards the
  // same space holds every wave's sums, [wave][ct][h][nt][lane] as f32x4
  constexpr int STAGE_U4 = kParts * 32 * K::PITCH, IDX_U4 = kDnSlots / 4;
  constexpr int PART_U4 = kParts * K::DT * 2 * NT * kWave;
  constexpr int BIG_U4 = STAGE_U4 + IDX_U4 > PART_U4 ? STAGE_U4 + IDX_U4 : PART_U4;
  __shared__ uint4 s_big[BIG_U4];
  __shared__ int s_wgrp[kBlock / kWave];
  __shared__ int2 s_ginfo[2 * kBlock + kDnPad];
  uint4* const s_stage = s_big;
  int* const s_idx = reinterpret_cast<int*>(s_big + STAGE_U4);
  f32x4_t* const s_part = reinterpret_cast<f32x4_t*>(s_big);

  const int S = (d + WCOLS - 1) / WCOLS;
  const int chunk = blockIdx.x / S, cgrp = blockIdx.x % S;
  const Split chunks(nseg, R), segs(d_ff, nseg);
  const int seg_lo = chunks.start(chunk), seg_hi = chunks.start(chunk + 1);
  const int nsc = seg_hi - seg_lo;  // <= kBlock, guaranteed by the host
  const int row_lo = segs.start(seg_lo);
  const int nslot = segs.start(seg_hi) - row_lo;  // <= kDnSlots, guaranteed by the host
  const int tid = threadIdx.x, lane = lane_id(), wave = uniform(tid / kWave);
  const int slot_w = wave % CW, phase = wave / CW;

  // segment tid of the chunk has (c > 0) + (c > 32) fragment groups; their places in
  // the group table come from two ballots and the per-wave totals
  const int c = tid < nsc ? seg_count[seg_lo + tid] : 0;
  const int srow = tid < nsc ? segs.start(seg_lo + tid) - row_lo : 0;
  {
    // eight loads in flight per thread before their LDS stores
    const Buf ib = make_buf(seg_idx + row_lo, 4u * (uint32_t)nslot);
    for (int o0 = 0; o0 < nslot; o0 += 8 * kBlock) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int o = o0 + u * kBlock + tid;
        v[u] = ldb32(ib, o < nslot ? 4u * (uint32_t)o : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int o = o0 + u * kBlock + tid;
        if (o < nslot) s_idx[o] = v[u];
      }
    }
  }
  const uint64_t has1 = __ballot(c > 0), has2 = __ballot(c > 32);
  if (lane == 0) s_wgrp[wave] = __popcll(has1) + __popcll(has2);
  __syncthreads();
  int gbase = 0, ngrp = 0;
#pragma unroll
  for (int w = 0; w < kBlock / kWave; ++w) {
    const int v = s_wgrp[w];
    gbase += w < wave ? v : 0;
    ngrp += v;
  }
  ngrp = uniform(ngrp);
  if (tid < nsc) {
    const int b = gbase + rank_in_mask(has1) + rank_in_mask(has2);
    const int zg = 2 * (seg_lo + tid);
    if (c > 0) s_ginfo[b] = make_int2(srow | (min(c, 32) << 16), zg);
    if (c > 32) s_ginfo[b + 1] = make_int2((srow + 32) | ((c - 32) << 16), zg + 1);
  }
  if (tid < kDnPad) s_ginfo[ngrp + tid] = make_int2(0, 0);
  __syncthreads();

  f32x4_t acc[K::DT][2][NT];
#pragma unroll
  for (int ct = 0; ct < K::DT; ++ct)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[ct][h][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // this lane's 16-byte chunk of the wave's columns
  const int ch = (cgrp * WCOLS + slot_w * 32 * K::DT) / W::EPC + lane % K::LPR;
  if (phase < ngrp) {
    // two register sets alternate, one group each per half-iteration; the table entry of
    // group j + 3 GS and the slot indices of group j + 2 GS are read while group j is
    // multiplied.  A pair always multiplies both halves (a group past the last one loads
    // nothing and adds zeros), so no load sits on a conditional path.
    DnFrags<NT, W> f0, f1;
    DnRows<NT, W> a = dn_rows<NT, W>(s_ginfo[phase], s_idx, C, ch);
    dn_issue(f0, a, db, zb, C, ch, T, ntt);
    a = dn_rows<NT, W>(s_ginfo[phase + GS], s_idx, C, ch);
    int2 info = s_ginfo[phase + 2 * GS];
    for (int j = phase;; j += 2 * GS) {
      dn_issue(f1, a, db, zb, C, ch, T, ntt);
      issue_barrier();
      a = dn_rows<NT, W>(info, s_idx, C, ch);
      info = s_ginfo[j + 3 * GS];
      dn_mma(f0, s_stage + wave * 32 * K::PITCH, acc);
      dn_issue(f0, a, db, zb, C, ch, T, ntt);
      issue_barrier();
      a = dn_rows<NT, W>(info, s_idx, C, ch);
      info = s_ginfo[j + 4 * GS];
      dn_mma(f1, s_stage + wave * 32 * K::PITCH, acc);
      if (j + 2 * GS >= ngrp) break;
    }
  }
  // lane m + 16 g of wave w holds tokens 16 nt + 4g .. + 3 of column 32 ct + 16 h + m
  // of slot w % CW; the GS waves of a slot are added in a fixed order, then one fp32
  // atomic per token and column goes to y
  __syncthreads();  // every wave is done with its tile and the slot indices
#pragma unroll
  for (int ct = 0; ct < K::DT; ++ct)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) s_part[(((wave * K::DT + ct) * 2 + h) * NT + nt) * kWave + lane] = acc[ct][h][nt];
  __syncthreads();
  constexpr int NE = CW * K::DT * 2 * NT * kWave;
  for (int o = tid; o < NE; o += kBlock) {
    const int l = o % kWave, r = o / kWave;  // r = ((slot DT + ct) 2 + h) NT + nt
    const int nt = r % NT, h = (r / NT) % 2, ct = (r / (2 * NT)) % K::DT, slot = r / (2 * NT * K::DT);
    const int tok0 = 16 * nt + 4 * (l >> 4);
    const int col = cgrp * WCOLS + slot * 32 * K::DT + 32 * ct + 16 * h + (l & 15);
    if (tok0 >= T || col >= d) continue;
    f32x4_t v = s_part[(((slot * K::DT + ct) * 2 + h) * NT + nt) * kWave + l];
#pragma unroll
    for (int p = 1; p < GS; ++p) v += s_part[((((slot + CW * p) * K::DT + ct) * 2 + h) * NT + nt) * kWave + l];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (tok0 + i < T) unsafeAtomicAdd(y + (size_t)(tok0 + i) * d + col, v[i]);
  }
}

// ------------------------------------------------------------------ host side
int token_tiles(const Workspace& ws) { return (ws.tc + 15) / 16; }

hipError_t split_tokens(const Shape& sh, const float* x, const Workspace& ws, hipStream_t s) {
  const int C = sh.d / 8, nks = (C + 3) / 4, ntt = token_tiles(ws);
  const int n = nks * ntt * kWave;
  k_split_tokens<<<(n + kBlock - 1) / kBlock, kBlock, 0, s>>>(x, C, sh.T, nks, ntt, ws.xs);
  return hipGetLastError();
}
template <class W, int NT, bool PRE>
hipError_t z_mfma(const Shape& sh, const Form& form, const float* x, const void* lopa_a, const Workspace& ws,
                  hipStream_t s) {
  const int C = sh.d / 8, ngrp = PRE ? token_tiles(ws) / NT : 1, grid = ((sh.r + 15) / 16) * kZParts * ngrp;
  // with G, extra workgroups write G x for the gate kernel
  const GWork gw{form, x, ws.gx, sh.T, sh.d, sh.d_ff, grid};
  const int g = grid + (form.g_idx ? (g_items(sh.d_ff, sh.T) + kZWaves * kWave - 1) / (kZWaves * kWave) : 0);
  k_lopa_z_mfma<NT, PRE, W><<<g, kZWaves * kWave, 0, s>>>(x, ws.xs, token_tiles(ws), static_cast<const uint4*>(lopa_a),
                                                      C, sh.T, sh.r, ws.tc, ws.z, gw, sh.sc.a);
  return hipGetLastError();
}

// Row-balanced segments of at most 64 rows; beyond 128 of them the count is a multiple
// of the gate kernel's grid so that every workgroup gets the same number.
int segments_for(int d_ff, int grid) {
  const int n = (d_ff + kSegRowsB - 1) / kSegRowsB;
  return n > 128 ? (n + grid - 1) / grid * grid : n;
}

// The 4x4x4 kernel takes batches of at most four tokens whose rows (and LoPA's r), padded to
// a whole step, fit its token LDS.
template <class W>
bool q4_fits(const Shape& sh, bool lopa) {
  const int step = 16 * W::EPC;
  return sh.T <= 4 && (sh.d + step - 1) / step * step <= kQ4MaxX && (!lopa || (sh.r + step - 1) / step * step <= kQ4MaxZ);
}

template <class W, bool LOPA, bool DENSE, int NT, int FORM>
hipError_t gate_mfma(const Shape& sh, const Form& form, const float* x, const void* gate_w, const void* w_up, float t,
                     Workspace& ws, float* y, hipStream_t s) {
  const int Cu = sh.d / 8, Cg = LOPA ? sh.r / 8 : Cu;
  if constexpr (NT == 1)
    if (q4_fits<W>(sh, LOPA)) {
      ws.nseg = segments_for(sh.d_ff, kSegGrid);
      return launch_gate_kernel_n(k_gate_up_q4<W, LOPA, DENSE, FORM>, ws.nseg < kSegGrid ? ws.nseg : kSegGrid,
                                  kQ4Threads, s, x,
                                (const float*)ws.z, static_cast<const uint4*>(gate_w), Cg,
                                static_cast<const uint4*>(w_up), Cu, sh.T, sh.d, sh.d_ff, ws.nseg, t, ws.slots, ws.tc,
                                ws.meta, ws.seg_count, ws.seg_idx, ws.seg_act, ws.zf, y, ws.xs, token_tiles(ws), form,
                                (const float*)ws.gx, LOPA ? sh.sc.b : sh.sc.gate, sh.sc.up, sh.sc.down);
    }
  // two workgroups a CU only where their segments stay near 64 rows: halving 8B-shaped
  // segments to 28 rows left the row tiles half empty (int8 / int4 at four tokens: 52.7 /
  // 54.4 us a call, 42.1 / 41.9 us with one workgroup a CU).  On the 70B shape LoPA gains
  // too (eight tokens: gate kernel 76.1 -> 71.1 us), where one workgroup a CU walks two
  // segments one after the other.
  const bool two = NT == 1 && sh.d_ff >= 48 * kSegGrid2;
  const int grid = two ? kSegGrid2 : kSegGrid;
  ws.nseg = segments_for(sh.d_ff, grid);
  const int g = ws.nseg < grid ? ws.nseg : grid;
  auto kernel = k_gate_up_mfma<W, LOPA, DENSE, NT, FORM>;
  if constexpr (NT == 1)
    if (two) kernel = k_gate_up_mfma2<W, LOPA, DENSE, FORM>;
  return launch_gate_kernel(kernel, g, s, x, (const float*)ws.z, static_cast<const uint4*>(gate_w), Cg,
                            static_cast<const uint4*>(w_up), Cu, sh.T, sh.d, sh.d_ff, ws.nseg, t, ws.slots, ws.tc,
                            ws.meta, ws.seg_count, ws.seg_idx, ws.seg_act, ws.zf, y, ws.xs, token_tiles(ws), form,
                            (const float*)ws.gx, LOPA ? sh.sc.b : sh.sc.gate, sh.sc.up, sh.sc.down);
}

template <class W, bool LOPA, bool DENSE, int FORM>
hipError_t gate_nt(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up, float t,
                   Workspace& ws, float* y, hipStream_t s) {
  if (sh.T <= 16) return gate_mfma<W, LOPA, DENSE, 1, FORM>(sh, f, x, gate_w, w_up, t, ws, y, s);
  if (sh.T <= 32) return gate_mfma<W, LOPA, DENSE, 2, FORM>(sh, f, x, gate_w, w_up, t, ws, y, s);
  return gate_mfma<W, LOPA, DENSE, 4, FORM>(sh, f, x, gate_w, w_up, t, ws, y, s);
}

template <class W, bool LOPA, bool DENSE>
hipError_t gate_form(const Shape& sh, const Form& f, const float* x, const void* gate_w, const void* w_up, float t,
                     Workspace& ws, float* y, hipStream_t s) {
  // the norm runs before this kernel, so only G needs the LoPA form here
  if constexpr (LOPA)
    if (f.g_idx) return gate_nt<W, LOPA, DENSE, kFormLoPA>(sh, f, x, gate_w, w_up, t, ws, y, s);
  return f.full() ? gate_nt<W, LOPA, DENSE, kFormAct>(sh, f, x, gate_w, w_up, t, ws, y, s)
                  : gate_nt<W, LOPA, DENSE, kFormDefault>(sh, f, x, gate_w, w_up, t, ws, y, s);
}

// Down grid: S column groups x R row chunks, about kDnWgTarget workgroups, at most
// kDnAtomicsMax fp32 atomics into y (fewer, longer row chunks measured faster than more
// parallel short ones), every chunk within the LDS slot and segment limits.
constexpr int kDnWgTarget = 512;
constexpr int64_t kDnAtomicsMax = 1 << 20;

template <class W, int NT>
hipError_t down_mfma(const Shape& sh, const void* w_down_t, const Workspace& ws, float* y, hipStream_t s) {
  const int C = sh.d / W::EPC;
  const int64_t wcols = DnCfg<NT, W>::WCOLS;
  const int64_t S = ((int64_t)sh.d + wcols - 1) / wcols;
  int64_t R = (kDnWgTarget + S - 1) / S;
  const int64_t amax = kDnAtomicsMax / ((int64_t)sh.T * sh.d);
  if (R > amax) R = amax;
  const int64_t rmin = (ws.nseg + kBlock - 1) / kBlock;
  if (R < rmin) R = rmin;
  if (R > ws.nseg) R = ws.nseg;
  if (R < 1) R = 1;
  const int64_t rows_per_seg = (sh.d_ff + ws.nseg - 1) / ws.nseg;
  while (R < ws.nseg && ((ws.nseg + R - 1) / R) * rows_per_seg > kDnSlots) ++R;
  if (((ws.nseg + R - 1) / R) * rows_per_seg > kDnSlots || S * R > INT32_MAX) return hipErrorInvalidValue;
  k_down_mfma<NT, W><<<(int)(S * R), kBlock, 0, s>>>(ws.seg_count, ws.seg_idx, ws.zf, ws.nseg, sh.d_ff, (int)R,
                                                     ws.tc, static_cast<const uint4*>(w_down_t), C, sh.d, sh.T, y);
  return hipGetLastError();
}

// One call of the path for weights of format W (after the tokens are split, if they are).
template <class W>
hipError_t batched_format(const Shape& sh, Gate g, bool dense, const Form& form, const float* x, const void* lopa_a,
                          const void* gate_w, const void* w_up, const void* w_down_t, float t, Workspace& ws,
                          float* y, hipStream_t s) {
  const bool lopa = g == Gate::LoPA;
  hipError_t e = hipSuccess;
  if (lopa) {
    // pre-split tokens (more than 16): one token tile a workgroup
    e = sh.T <= 16 ? z_mfma<W, 1, false>(sh, form, x, lopa_a, ws, s) : z_mfma<W, 1, true>(sh, form, x, lopa_a, ws, s);
    if (e != hipSuccess) return e;
    // RMSNorm between A and B: the two partial copies of z become one normalised copy
    if (form.rms_eps > 0.f &&
        (e = launch_rms_norm(ws.z, 2, ws.tc, sh.T, sh.r, form.rms_gain, form.rms_eps, s)) != hipSuccess)
      return e;
  }
  if (lopa)
    e = dense ? gate_form<W, true, true>(sh, form, x, gate_w, w_up, t, ws, y, s)
              : gate_form<W, true, false>(sh, form, x, gate_w, w_up, t, ws, y, s);
  else
    e = dense ? gate_form<W, false, true>(sh, form, x, gate_w, w_up, t, ws, y, s)
              : gate_form<W, false, false>(sh, form, x, gate_w, w_up, t, ws, y, s);
  if (e != hipSuccess) return e;
  if (sh.T <= 16) return down_mfma<W, 1>(sh, w_down_t, ws, y, s);
  if (sh.T <= 32) return down_mfma<W, 2>(sh, w_down_t, ws, y, s);
  return down_mfma<W, 4>(sh, w_down_t, ws, y, s);
}

}  // namespace

// The matrix-core path addresses every operand with 32-bit byte offsets below 2^31.
// bf16 weights, and int8 / int4 codes (converted to bf16 on their way into the operand
// tiles): rows of whole 16-byte chunks, so d (and LoPA's r) a multiple of 16 / 32.
bool batched_ok(const Shape& sh, Gate g) {
  if (sh.wdt < 1 || sh.wdt > 3 || sh.T < 2 || sh.T > kTokChunk) return false;
  const int q = sh.wdt == 1 ? 8 : sh.wdt == 2 ? 16 : 32;  // elements a 16-byte chunk
  if (sh.d % q != 0) return false;
  const int64_t lim = int64_t(1) << 31;
  if (2 * (int64_t)sh.d_ff * sh.d >= lim || 4 * (int64_t)kTokChunk * sh.d >= lim) return false;
  if ((int64_t)segments_for(sh.d_ff, kSegGrid2) * 256 * kTokChunk >= lim) return false;
  if (g == Gate::LoPA && (sh.r % q != 0 || 2 * (int64_t)sh.d_ff * sh.r >= lim || 2 * (int64_t)sh.r * sh.d >= lim ||
                          4 * (int64_t)kTokChunk * sh.d_ff >= lim))  // G x, read through a buffer
    return false;
  return true;
}

// the most segments any gate kernel of this path uses (workspace sizing)
int batched_segments(int d_ff) { return segments_for(d_ff, kSegGrid2); }

hipError_t launch_batched(const Shape& sh, Gate g, bool dense, const Form& form, const float* x,
                          const void* lopa_a, const void* gate_w, const void* w_up, const void* w_down_t, float t,
                          Workspace& ws, float* y, hipStream_t s) {
  hipError_t e = hipSuccess;
  // more than one token tile: the kernels read the tokens pre-split
  if (sh.T > 16 && (e = split_tokens(sh, x, ws, s)) != hipSuccess) return e;
  if (sh.wdt == 2) return batched_format<WI8>(sh, g, dense, form, x, lopa_a, gate_w, w_up, w_down_t, t, ws, y, s);
  if (sh.wdt == 3) return batched_format<WI4>(sh, g, dense, form, x, lopa_a, gate_w, w_up, w_down_t, t, ws, y, s);
  return batched_format<WBf16>(sh, g, dense, form, x, lopa_a, gate_w, w_up, w_down_t, t, ws, y, s);
}


}  // namespace ffn

// gfx950 kernels for a batch of 2..64 tokens with bf16 weights (paper Section 5.3: the
// rows of W_up / W_down are read once for the union of the tokens' active sets).
//
// The gate (W_gate x or B z), the W_up dots of the union rows and LoPA's A x are
// dense contractions over a token tile, so they run on the matrix cores:
// v_mfma_f32_16x16x32_bf16 with a 16-row weight tile as the A operand and 16 tokens as
// the B operand.  The fp32 tokens are split into bf16 hi + lo (x - hi rounded again),
// two MFMAs per step: the products are exact in fp32 and the split leaves a relative
// error of about 2^-16 on each token element, far inside the 1e-3 band of the active
// set decision.  Weights are read straight from HBM into the A operand: lane l holds
// 8 consecutive bf16 of row (l mod 16); the four lane groups l / 16 take four
// consecutive 16-byte chunks, so one instruction reads 64 contiguous bytes of each of
// 16 rows.  Which k positions a lane group holds does not matter for a full
// reduction as long as the A and B operands use the same ones.
//
// The down projection accumulates zval[tau][k] * w_down_t[idx_k] for 2..8 tokens on
// the vector ALUs (every weight element feeds T FMAs), 128 columns per workgroup.  For
// 9..64 tokens it is a matrix-core product Y[tokens][cols] = Z[tokens][entries] x
// D[entries][cols] whose reduction runs over the gathered rows.  The B operand needs 8
// entries of one column per lane, but a row gather gives a lane 8 columns of one entry;
// an MFMA against a 0/1 selector matrix transposes each 16 x 16 block exactly in fp32
// (every output is one weight times 1), and its output layout (lane = column,
// lane group = entries 4g..4g+3) is already the B-operand layout of the product.
#include "ffn_device.h"
#include "ffn_internal.h"

namespace ffn {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kMRows = 32;  // gate rows per segment of the batched gate kernel (two 16-row tiles)
constexpr int kKU = 8;      // k steps (32 elements each) loaded per unrolled group

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// x = hi + lo with both in bf16 (round to nearest even twice)
__device__ __forceinline__ void split_bf16(const float (&v)[8], bf16x8_t& hi, bf16x8_t& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const __bf16 h = (__bf16)v[j];
    hi[j] = h;
    lo[j] = (__bf16)(v[j] - (float)h);
  }
}

// B operand of one k step: 8 consecutive elements (chunk c) of token `tok`'s vector,
// split into hi / lo; zero outside the batch or the row.
__device__ __forceinline__ void vec_frag(const float* __restrict__ vec, int len, int T, int tok, int c, int C,
                                         bf16x8_t& hi, bf16x8_t& lo) {
  float v[8];
  if (tok < T && c < C) {
    const float4* p = reinterpret_cast<const float4*>(vec + (size_t)tok * len + (size_t)c * 8);
    const float4 a = p[0], b = p[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = 0.f;
  }
  split_bf16(v, hi, lo);
}

// acc[nt] += (16 rows starting at this lane's row) . (tokens 16 nt .. 16 nt + 15) over
// k steps [ks0, ks1); a k step covers chunks 4 ks .. 4 ks + 3 of the rows.
template <int NT>
__device__ __forceinline__ void mfma_rows(const uint4* __restrict__ wrow, bool rok, int C,
                                          const float* __restrict__ vec, int len, int T, int ks0, int ks1,
                                          f32x4_t (&acc)[NT]) {
  const int lane = lane_id(), m = lane & 15, g = lane >> 4;
  for (int ks = ks0; ks < ks1; ks += kKU) {
    uint4 a[kKU];
#pragma unroll
    for (int u = 0; u < kKU; ++u) {
      const int c = (ks + u) * 4 + g;
      a[u] = (rok && ks + u < ks1 && c < C) ? ld_weights(wrow + c) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kKU; ++u) {
      if (ks + u < ks1) {
        const int c = (ks + u) * 4 + g;
        const bf16x8_t av = __builtin_bit_cast(bf16x8_t, a[u]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          bf16x8_t hi, lo;
          vec_frag(vec, len, T, nt * 16 + m, c, C, hi, lo);
          acc[nt] = mfma16(av, hi, acc[nt]);
          acc[nt] = mfma16(av, lo, acc[nt]);
        }
      }
    }
  }
}

// k-step range of k part kp out of np for rows of C chunks
__device__ __forceinline__ void kpart(int C, int kp, int np, int* ks0, int* ks1) {
  const int nks = (C + 3) / 4;
  const int per = (nks + np - 1) / np;
  *ks0 = min(nks, kp * per);
  *ks1 = min(nks, *ks0 + per);
}

// ------------------------------------------------------------------ gate + W_up
// One segment of <= 32 neurons per workgroup.  Wave w computes row tile w & 1 over
// half w >> 1 of the k range; the halves are added through LDS.  A neuron joins the
// union if any token activates it; one ballot orders the union; the W_up dots of the
// union rows (tiles of 16 gathered rows, same k split) give zval = act * v per token.
template <bool LOPA, bool DENSE, int NT>
__global__ __launch_bounds__(kBlock) void k_gate_up_mfma(const float* __restrict__ x, const float* __restrict__ z,
                                                         const uint4* __restrict__ gate_w, int Cg,
                                                         const uint4* __restrict__ w_up, int Cu, int T, int d, int r,
                                                         int d_ff, int nseg, float t, int slots,
                                                         int32_t* __restrict__ meta, int32_t* __restrict__ seg_count,
                                                         int32_t* __restrict__ seg_idx, float* __restrict__ seg_act,
                                                         float* __restrict__ seg_zval, float* __restrict__ y) {
  __shared__ f32x4_t s_part[2][NT][kWave];
  __shared__ float s_act[kMRows][kTokChunk];
  __shared__ uint32_t s_mask[2];
  __shared__ int s_list[kMRows];
  __shared__ int s_cnt;

  const int seg = blockIdx.x;
  const int row0 = seg_row(seg, d_ff, nseg);
  const int nrows = seg_row(seg + 1, d_ff, nseg) - row0;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int m = lane & 15, g = lane >> 4;
  const int tile = wave & 1, kp = wave >> 1;
  clear_output(y, T * d, meta, nseg);

  // gate values h[row][token]
  f32x4_t acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  {
    const int rl = tile * 16 + m;
    const bool rok = rl < nrows;
    int ks0, ks1;
    kpart(Cg, kp, 2, &ks0, &ks1);
    mfma_rows<NT>(gate_w + (size_t)(row0 + (rok ? rl : 0)) * Cg, rok, Cg, LOPA ? z : x, LOPA ? r : d, T, ks0, ks1,
                  acc);
  }
  if (kp == 1)
    for (int nt = 0; nt < NT; ++nt) s_part[tile][nt][lane] = acc[nt];
  __syncthreads();
  if (kp == 0) {
    // lane holds h of rows tile*16 + 4g + i (i < 4) for tokens 16 nt + m
    uint32_t mask = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rl = tile * 16 + 4 * g + i;
      bool any = false;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float h = acc[nt][i] + s_part[tile][nt][lane][i];
        const int tok = nt * 16 + m;
        const bool on = tok < T && h > t;  // NaN compares false: inactive
        if (tok < T && rl < nrows) s_act[rl][tok] = on ? h - t : 0.f;
        any |= on;
      }
      const uint64_t b = __ballot(any && rl < nrows);
#pragma unroll
      for (int gg = 0; gg < 4; ++gg)
        if ((b >> (16 * gg)) & 0xffffull) mask |= 1u << (4 * gg + i);
    }
    if (lane == 0) s_mask[tile] = mask;
  }
  __syncthreads();

  // ascending union of the segment
  if (wave == 0) {
    const uint32_t on = s_mask[0] | (s_mask[1] << 16);
    const bool sel = lane < nrows && (DENSE || ((on >> lane) & 1u));
    const uint64_t b = __ballot(sel);
    const int rank = rank_in_mask(b);
    if (sel) {
      s_list[rank] = lane;
      seg_idx[row0 + rank] = row0 + lane;
      for (int tok = 0; tok < T; ++tok) seg_act[(size_t)tok * slots + row0 + rank] = s_act[lane][tok];
    }
    if (lane == 0) {
      s_cnt = __popcll(b);
      seg_count[seg] = s_cnt;
    }
  }
  __syncthreads();

  // W_up dots of the union rows: tiles of 16 entries
  const int cnt = s_cnt;
  const bool tile_on = tile * 16 < cnt;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if (tile_on) {
    const int e = tile * 16 + m;
    const bool eok = e < cnt;
    int ks0, ks1;
    kpart(Cu, kp, 2, &ks0, &ks1);
    mfma_rows<NT>(w_up + (size_t)(row0 + (eok ? s_list[e] : 0)) * Cu, eok, Cu, x, d, T, ks0, ks1, acc);
    if (kp == 1)
      for (int nt = 0; nt < NT; ++nt) s_part[tile][nt][lane] = acc[nt];
  }
  __syncthreads();
  if (tile_on && kp == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tile * 16 + 4 * g + i;
      if (e < cnt) {
        const int kr = s_list[e];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int tok = nt * 16 + m;
          if (tok < T)
            seg_zval[(size_t)tok * slots + row0 + e] = s_act[kr][tok] * (acc[nt][i] + s_part[tile][nt][lane][i]);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ LoPA z = A x
// One 16-row tile of A per workgroup of kZWaves waves, each over 1/kZWaves of d.
constexpr int kZWaves = 8;

template <int NT>
__global__ __launch_bounds__(kZWaves * kWave) void k_lopa_z_mfma(const float* __restrict__ x,
                                                                 const uint4* __restrict__ A, int C, int T, int d,
                                                                 int r, float* __restrict__ z) {
  __shared__ f32x4_t s_part[kZWaves][NT][kWave];
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int m = lane & 15, g = lane >> 4;
  const int row = blockIdx.x * 16 + m;
  const bool rok = row < r;
  f32x4_t acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  int ks0, ks1;
  kpart(C, wave, kZWaves, &ks0, &ks1);
  mfma_rows<NT>(A + (size_t)(rok ? row : 0) * C, rok, C, x, d, T, ks0, ks1, acc);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) s_part[wave][nt][lane] = acc[nt];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4_t s = s_part[0][nt][lane];
      for (int w = 1; w < kZWaves; ++w) s += s_part[w][nt][lane];
      const int tok = nt * 16 + m;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = blockIdx.x * 16 + 4 * g + i;
        if (tok < T && k < r) z[(size_t)tok * r + k] = s[i];
      }
    }
  }
}

// ------------------------------------------------------------------ down, 2..8 tokens
// Workgroup b: row chunk b / S (segments [c nseg/R, (c+1) nseg/R)), column slice b % S
// of 16 chunks (128 bf16 columns).  A wave instruction reads 256 bytes of each of 4
// rows.  The chunk's ascending active list is staged in LDS a window at a time, with
// the per-token zval of each entry; partial sums go to y with fp32 atomics.
constexpr int kDnSliceChunks = 16;
constexpr int kDnWindow = 512;

template <int TT>
__global__ __launch_bounds__(kBlock) void k_down_tn(const int32_t* __restrict__ seg_count,
                                                    const int32_t* __restrict__ seg_idx,
                                                    const float* __restrict__ seg_zval, int nseg, int d_ff, int R,
                                                    int slots, const uint4* __restrict__ w_down_t, int C, int d, int T,
                                                    float* __restrict__ y) {
  constexpr int U = 8, kWaves = kBlock / kWave, RPW = kWave / kDnSliceChunks;  // rows per wave load
  __shared__ int s_off[kBlock + 1];
  __shared__ int s_idx[kDnWindow];
  __shared__ float s_z[TT][kDnWindow];
  __shared__ float s_red[kWaves][kDnSliceChunks][TT][8];

  const int S = (C + kDnSliceChunks - 1) / kDnSliceChunks;
  const int chunk = blockIdx.x / S, slice = blockIdx.x % S;
  const int seg_lo = (int)(((int64_t)chunk * nseg) / R), seg_hi = (int)(((int64_t)(chunk + 1) * nseg) / R);
  const int nsc = seg_hi - seg_lo;  // <= kBlock, guaranteed by the host
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int q = lane % kDnSliceChunks, p = lane / kDnSliceChunks;

  s_off[threadIdx.x] = threadIdx.x < nsc ? seg_count[seg_lo + threadIdx.x] : 0;
  __syncthreads();
  block_exclusive_scan(s_off, kBlock);
  const int n = s_off[kBlock];

  const int ch = slice * kDnSliceChunks + q;
  const bool cvalid = ch < C;
  float acc[TT][8];
#pragma unroll
  for (int tau = 0; tau < TT; ++tau)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[tau][e] = 0.f;

  for (int base = 0; base < n; base += kDnWindow) {
    const int wn = min(kDnWindow, n - base);
    // stage entries [base, base + wn): binary search of the owning segment
    for (int k = threadIdx.x; k < wn; k += kBlock) {
      const int kk = base + k;
      int lo = 0, hi = nsc - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= kk) lo = mid; else hi = mid - 1;
      }
      const int slot = seg_row(seg_lo + lo, d_ff, nseg) + (kk - s_off[lo]);
      s_idx[k] = seg_idx[slot];
      for (int tau = 0; tau < TT; ++tau) s_z[tau][k] = tau < T ? seg_zval[(size_t)tau * slots + slot] : 0.f;
    }
    __syncthreads();
    for (int k = wave * RPW + p; k < wn; k += kWaves * RPW * U) {
      uint4 wv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kk = k + u * kWaves * RPW;
        wv[u] = (kk < wn && cvalid) ? ld_weights(w_down_t + (size_t)s_idx[kk] * C + ch) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kk = k + u * kWaves * RPW;
        if (kk < wn) {
          float f[8];
          unpack(WBf16{}, wv[u], f);
#pragma unroll
          for (int tau = 0; tau < TT; ++tau) {
            const float zz = s_z[tau][kk];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[tau][e] = fmaf(zz, f[e], acc[tau][e]);
          }
        }
      }
    }
    __syncthreads();
  }

  // reduce over the 4 row lanes of a wave (lane bits 4, 5), then over the waves
#pragma unroll
  for (int tau = 0; tau < TT; ++tau)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = acc[tau][e];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      acc[tau][e] = v;
    }
  if (p == 0)
#pragma unroll
    for (int tau = 0; tau < TT; ++tau)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_red[wave][q][tau][e] = acc[tau][e];
  __syncthreads();
  for (int o = threadIdx.x; o < kDnSliceChunks * TT * 8; o += kBlock) {
    const int e = o % 8, tau = (o / 8) % TT, qq = o / (8 * TT);
    if (tau >= T) continue;
    float s = s_red[0][qq][tau][e];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) s += s_red[w][qq][tau][e];
    const int col = (slice * kDnSliceChunks + qq) * 8 + e;
    if (col < d) unsafeAtomicAdd(y + (size_t)tau * d + col, s);
  }
}

// ------------------------------------------------------------------ down, 9..64 tokens
// Workgroup b: 128-column group b % S4 (S4 = ceil(C / 16)), row chunk b / S4; wave w
// owns the 32 columns w of the group.  The chunk's slot list is expanded into LDS once;
// then kMdWindow entries at a time the row indices and per-token zvals are staged and
// every wave issues all its W_down loads of the window before the matrix-core work.
// Partial sums over the R row chunks go to y with fp32 atomics.
constexpr int kMdWindow = 128;
constexpr int kMdChunkMax = 4096;  // most active entries of one row chunk

template <int NT>
__global__ __launch_bounds__(kBlock) void k_down_mfma(const int32_t* __restrict__ seg_count,
                                                      const int32_t* __restrict__ seg_idx,
                                                      const float* __restrict__ seg_zval, int nseg, int d_ff, int R,
                                                      int slots, const uint4* __restrict__ w_down_t, int C, int d,
                                                      int T, float* __restrict__ y) {
  constexpr int KG = kMdWindow / 32;  // 32-entry k groups per window
  __shared__ int s_off[kBlock + 1];
  __shared__ int s_slot[kMdChunkMax];
  __shared__ int s_idx[kMdWindow];
  __shared__ float s_z[NT * 16][kMdWindow + 4];

  const int S4 = (C + 15) / 16;
  const int chunk = blockIdx.x / S4, cgrp = blockIdx.x % S4;
  const int seg_lo = (int)(((int64_t)chunk * nseg) / R), seg_hi = (int)(((int64_t)(chunk + 1) * nseg) / R);
  const int nsc = seg_hi - seg_lo;  // <= kBlock, guaranteed by the host
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  const int m = lane & 15, g = lane >> 4;
  const int ch = cgrp * 16 + wave * 4 + g;  // this lane's 8 columns in the transposition tiles
  const bool cvalid = ch < C;

  s_off[threadIdx.x] = threadIdx.x < nsc ? seg_count[seg_lo + threadIdx.x] : 0;
  __syncthreads();
  block_exclusive_scan(s_off, kBlock);
  const int n = min(s_off[kBlock], kMdChunkMax);
  if (threadIdx.x < nsc) {
    const int k0 = s_off[threadIdx.x], k1 = min(s_off[threadIdx.x + 1], kMdChunkMax);
    const int slot0 = seg_row(seg_lo + threadIdx.x, d_ff, nseg);
    for (int k = k0; k < k1; ++k) s_slot[k] = slot0 + (k - k0);
  }

  // 0/1 selectors: column 16 h + m of the 32-column tile
  bf16x8_t sel[2];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int j = 0; j < 8; ++j) sel[h][j] = (__bf16)((8 * g + j == 16 * h + m) ? 1.f : 0.f);

  f32x4_t acc[2][NT];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[h][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int base = 0; base < n; base += kMdWindow) {
    const int wn = min(kMdWindow, n - base);
    __syncthreads();  // slot list ready / previous window consumed
    for (int o = threadIdx.x; o < kMdWindow * (NT * 16 + 1); o += kBlock) {
      const int k = o % kMdWindow, row = o / kMdWindow;  // row 0: index, rows 1..: tokens
      const bool ok = k < wn;
      const int slot = ok ? s_slot[base + k] : 0;
      if (row == 0) {
        s_idx[k] = ok ? seg_idx[slot] : 0;
      } else {
        const int tau = row - 1;
        s_z[tau][k] = (ok && tau < T) ? seg_zval[(size_t)tau * slots + slot] : 0.f;
      }
    }
    __syncthreads();
    uint4 a[KG][2];
#pragma unroll
    for (int kg = 0; kg < KG; ++kg)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int e = kg * 32 + hh * 16 + m;
        a[kg][hh] = (e < wn && cvalid) ? ld_weights(w_down_t + (size_t)s_idx[e] * C + ch) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
    for (int kg = 0; kg < KG; ++kg) {
      if (kg * 32 >= wn) break;
      const bf16x8_t t0 = __builtin_bit_cast(bf16x8_t, a[kg][0]), t1 = __builtin_bit_cast(bf16x8_t, a[kg][1]);
      bf16x8_t bfrag[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
        const f32x4_t c0 = mfma16(t0, sel[h], zero);  // entries 4g..4g+3 of column 16h + m
        const f32x4_t c1 = mfma16(t1, sel[h], zero);  // entries 16+4g..16+4g+3
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bfrag[h][j] = (__bf16)c0[j];
          bfrag[h][4 + j] = (__bf16)c1[j];
        }
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float* zr = &s_z[nt * 16 + m][kg * 32];
        float v[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[j] = zr[4 * g + j];
          v[4 + j] = zr[16 + 4 * g + j];
        }
        bf16x8_t zhi, zlo;
        split_bf16(v, zhi, zlo);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          acc[h][nt] = mfma16(zhi, bfrag[h], acc[h][nt]);
          acc[h][nt] = mfma16(zlo, bfrag[h], acc[h][nt]);
        }
      }
    }
  }

#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int col = (cgrp * 16 + wave * 4) * 8 + 16 * h + m;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tau = nt * 16 + 4 * g + i;
        if (tau < T && col < d) unsafeAtomicAdd(y + (size_t)tau * d + col, acc[h][nt][i]);
      }
  }
}

}  // namespace

// ------------------------------------------------------------------ launchers
bool batched_ok(const Shape& sh, Gate g) {
  if (sh.wdt != 1 || sh.T < 2 || sh.T > kTokChunk || sh.d % 8 != 0) return false;
  if (g == Gate::LoPA && sh.r % 8 != 0) return false;
  return true;
}

bool batched_down_ok(const Shape& sh) { return sh.wdt == 1 && sh.T >= 2 && sh.T <= kTokChunk && sh.d % 8 == 0; }

int batched_segments(int d_ff) { return (d_ff + kMRows - 1) / kMRows; }

hipError_t launch_lopa_z_batched(const Shape& sh, const float* x, const void* lopa_a, const Workspace& ws,
                                 hipStream_t s) {
  const int C = sh.d / 8, grid = (sh.r + 15) / 16;
  const uint4* A = static_cast<const uint4*>(lopa_a);
  if (sh.T <= 16)
    k_lopa_z_mfma<1><<<grid, kZWaves * kWave, 0, s>>>(x, A, C, sh.T, sh.d, sh.r, ws.z);
  else if (sh.T <= 32)
    k_lopa_z_mfma<2><<<grid, kZWaves * kWave, 0, s>>>(x, A, C, sh.T, sh.d, sh.r, ws.z);
  else
    k_lopa_z_mfma<4><<<grid, kZWaves * kWave, 0, s>>>(x, A, C, sh.T, sh.d, sh.r, ws.z);
  return hipGetLastError();
}

template <bool LOPA, bool DENSE>
hipError_t gate_up_batched(const Shape& sh, const float* x, const void* gate_w, const void* w_up, float t,
                           Workspace& ws, float* y, hipStream_t s) {
  ws.nseg = batched_segments(sh.d_ff);
  const int Cu = sh.d / 8, Cg = LOPA ? sh.r / 8 : Cu;
  const uint4* G = static_cast<const uint4*>(gate_w);
  const uint4* U = static_cast<const uint4*>(w_up);
#define FFN_GUB(NT)                                                                                              \
  return launch_gate_kernel(k_gate_up_mfma<LOPA, DENSE, NT>, ws.nseg, s, x, (const float*)ws.z, G, Cg, U, Cu, sh.T, \
                            sh.d, sh.r, sh.d_ff, ws.nseg, t, ws.slots, ws.meta, ws.seg_count, ws.seg_idx,         \
                            ws.seg_act, ws.seg_zval, y)
  if (sh.T <= 16) FFN_GUB(1);
  if (sh.T <= 32) FFN_GUB(2);
  FFN_GUB(4);
#undef FFN_GUB
}

hipError_t launch_gate_up_batched(const Shape& sh, Gate g, bool dense, const float* x, const void* gate_w,
                                  const void* w_up, float t, Workspace& ws, float* y, hipStream_t s) {
  if (g == Gate::LoPA)
    return dense ? gate_up_batched<true, true>(sh, x, gate_w, w_up, t, ws, y, s)
                 : gate_up_batched<true, false>(sh, x, gate_w, w_up, t, ws, y, s);
  return dense ? gate_up_batched<false, true>(sh, x, gate_w, w_up, t, ws, y, s)
               : gate_up_batched<false, false>(sh, x, gate_w, w_up, t, ws, y, s);
}

// about kDownAtomics fp32 atomics per call into y; at most kBlock segments per chunk
constexpr int64_t kDownAtomics = 512 * 1024;

hipError_t launch_down_batched(const Shape& sh, const void* w_down_t, const Workspace& ws, float* y, hipStream_t s) {
  const int C = sh.d / 8;
  const int S = (C + kDnSliceChunks - 1) / kDnSliceChunks;
  int R = (int)(kDownAtomics / ((int64_t)sh.T * sh.d));
  const int rmin = (ws.nseg + kBlock - 1) / kBlock;
  if (R < rmin) R = rmin;
  if (R > ws.nseg) R = ws.nseg;
  if (R < 1) R = 1;
  const uint4* D = static_cast<const uint4*>(w_down_t);
  if (sh.T > 8) {
    // row chunks: enough workgroups to cover the GPU, each chunk's rows fit the LDS slot list
    const int S4 = (C + 15) / 16;
    int Rm = (2 * 256 + S4 - 1) / S4;
    const int rows_per_seg = (sh.d_ff + ws.nseg - 1) / ws.nseg;
    const int rcap = (sh.d_ff + kMdChunkMax - 1) / kMdChunkMax + 1;
    if (Rm < rcap) Rm = rcap;
    if (Rm < rmin) Rm = rmin;
    while (Rm < ws.nseg && ((ws.nseg + Rm - 1) / Rm) * rows_per_seg > kMdChunkMax) ++Rm;
    if (Rm > ws.nseg) Rm = ws.nseg;
#define FFN_DM(NT)                                                                                                 \
  k_down_mfma<NT><<<S4 * Rm, kBlock, 0, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff, Rm, ws.slots, \
                                            D, C, sh.d, sh.T, y)
    if (sh.T <= 16)
      FFN_DM(1);
    else if (sh.T <= 32)
      FFN_DM(2);
    else
      FFN_DM(4);
#undef FFN_DM
    return hipGetLastError();
  }
  if (sh.T <= 2)
    k_down_tn<2><<<S * R, kBlock, 0, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff, R, ws.slots, D, C,
                                          sh.d, sh.T, y);
  else if (sh.T <= 4)
    k_down_tn<4><<<S * R, kBlock, 0, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff, R, ws.slots, D, C,
                                          sh.d, sh.T, y);
  else
    k_down_tn<8><<<S * R, kBlock, 0, s>>>(ws.seg_count, ws.seg_idx, ws.seg_zval, ws.nseg, sh.d_ff, R, ws.slots, D, C,
                                          sh.d, sh.T, y);
  return hipGetLastError();
}

}  // namespace ffn

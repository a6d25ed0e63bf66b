/*
 * ffn_oracle.c -- reference oracle for the activation-sparse gated FFN forward pass.
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg load this file's library.  It shares
 * no code, header, table or helper with the GPU library; it is deliberately plain
 * and slow: fp64 arithmetic, straight ascending loops, no blocking, no SIMD.
 *
 * What it computes (paper: "Model casting & Low-parameter gating: towards more
 * sparsely activated FFNs"):
 *
 *   Gated FFN, Section 3.1, Eq. (ffn):  y = W2 ( A(W1 x) (*) (W3 x) ),
 *     with W1 = W_gate, W3 = W_up, W2 = W_down; W2 is passed transposed
 *     (w_down_t[i][:] = column i of W2 = the output vector of hidden neuron i).
 *   Activation A: shifted ReLU, A(h) = max(h - t, 0) (the "shifted ReLU" of the
 *     activation ablation, Appendix M), so neuron i is active iff h_i > t.
 *   Exploitable zeros, Section 3.1 ("FFN FLOP-ratio"): a zero of A(W1 x) is known
 *     before W3 is applied, so the sparse method skips row i of W3 and column i
 *     of W2 for every inactive i, while W1 x is always computed in full.
 *   LoPA gating, Section 3.3, Eq. (lopaapprox): W1 = G + U V with U (H x r),
 *     V (r x D), V = lopa_a [r][d] and U = lopa_b [d_ff][r]: h = G x + U (V x).
 *     G has a single nonzero per row, +1 or -1 (Section 3.3 and the ablation of
 *     the fixed matrix): row i holds g_sign[i] in column g_idx[i], so
 *     (G x)_i = g_sign[i] * x[g_idx[i]].  Without g_idx / g_sign, G = 0.
 *     Optionally (Section 3.3, "LoPA in practice") an RMSNorm sits between the
 *     two factors: h = G x + U RMSNorm(V x), RMSNorm(z)_k = gain_k z_k /
 *     sqrt(mean_k z_k^2 + eps) over the r components.
 *   Zeros of the gated intermediate (the s_gated site of Table ffn-sparsity-sites,
 *     appendix on baseline details): a neuron whose value A(h) * v is exactly zero
 *     adds nothing, so the sparse method skips its column of W2 as well.  With the
 *     shifted ReLU or R-S+ on the gate and v or SiLU(v) on W3 this happens only
 *     where v is exactly zero.
 *   Activation variants (Section 3.1 "R-S+ activation"; Section 3.3 "Double
 *     activation"): act = 1 replaces the shifted ReLU by the shifted R-S+,
 *     A(h) = (h - t) sigma(h - t) for h > t and 0 otherwise (sigma the logistic
 *     function): the same active set, another value.  silu_up = 1 applies SiLU,
 *     v sigma(v), to the W3 output of each active neuron.
 *   FLOP accounting, Section 3.1 Eq. (flops_ratio) and Section 3.3: the oracle
 *     counts every multiply-add of the three matrix products it executes, so that
 *     the count can be compared with the paper's cost model: standard
 *     d*d_ff + 2|S|d, LoPA r(d + d_ff) + 2|S|d, dense 3 d d_ff (LoPA dense:
 *     r(d + d_ff) + 2 d d_ff).  Like the paper's model it leaves out G's gather
 *     and the norm.
 *
 * Inputs are exactly the bit patterns the GPU receives: x is fp32, weights are
 * fp32 (wdt = 0) or bfloat16 bit patterns (wdt = 1); both widen to double
 * exactly.  t is the same fp32 value, widened.
 *
 * Weight-only quantization (wdt = 2: int8, wdt = 3: int4; the setting of the
 * appendix on quantization-aware training, whose kernels read int8 or int4
 * weights at inference): the paper fixes no scheme, so one is chosen here.  Every
 * matrix row i carries a code row q_i and an fp32 scale s_i, and its weights are
 * s_i * q_ij, formed exactly in double.  int8 codes are signed bytes; int4 codes
 * are two's-complement nibbles, two per byte, element 2k in the low nibble of byte
 * k of the row (rows of even length).  The matrix rows are those of the stored
 * layout: W_gate, W3, V, U by output unit, W2 by hidden neuron (its transposed
 * rows).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

/* element k (in row `row`) of a weight matrix, widened exactly to double; for the
   quantized formats the row's scale times its code */
static double weight_at(const void* w, int wdt, const float* scale, size_t row, size_t k) {
  if (wdt == 0) return (double)((const float*)w)[k];
  if (wdt == 2) return (double)scale[row] * (double)((const int8_t*)w)[k];
  if (wdt == 3) {
    int b = ((const uint8_t*)w)[k >> 1];
    int q = (k & 1) ? (b >> 4) : (b & 15); /* element 2k in the low nibble */
    if (q >= 8) q -= 16;                   /* two's complement */
    return (double)scale[row] * (double)q;
  }
  uint32_t bits = ((uint32_t)((const uint16_t*)w)[k]) << 16; /* bf16 = top half of an fp32 */
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* <row i of an [n][len] matrix, v>, ascending j, counting multiply-adds */
static double row_dot(const void* w, int wdt, const float* scale, size_t i, int len, const double* v,
                      int64_t* macs) {
  double s = 0.0;
  for (int j = 0; j < len; ++j) s += weight_at(w, wdt, scale, i, i * (size_t)len + (size_t)j) * v[j];
  *macs += len;
  return s;
}

/* the logistic function 1 / (1 + e^-u) */
static double logistic(double u) { return 1.0 / (1.0 + exp(-u)); }

/*
 * oracle_ffn_q -- one FFN forward pass per token, tokens independent.
 *
 *   gating        0: standard, h = W_gate x          (w_gate [d_ff][d])
 *                 1: LoPA,     h = B (A x)           (lopa_a [r][d], lopa_b [d_ff][r])
 *   skip_inactive 1: the sparse method (inactive neurons' W_up rows and W_down
 *                    columns are never read)
 *                 0: the dense FFN (every neuron evaluated, inactive ones weigh 0)
 *   wdt           weight storage: 0 = fp32, 1 = bf16 bit patterns, 2 = int8 codes,
 *                 3 = int4 codes (row lengths d and r even)
 *   s_gate, s_a, s_b, s_up, s_down  int8 / int4 only: the fp32 row scales of
 *                 W_gate [d_ff], A [r], B [d_ff], W_up [d_ff], W_down^T [d_ff]
 *   x             [T][d] fp32
 *   t             activation threshold (shift of the activation)
 *   act           0: shifted ReLU, 1: shifted R-S+
 *   silu_up       1: SiLU on the W3 output (double activation)
 *   g_idx, g_sign LoPA only: G's column (in [0, d)) and value (+1 / -1) per row,
 *                 both NULL for G = 0
 *   rms_norm      LoPA only: 1 for h = G x + U RMSNorm(V x)
 *   rms_gain      [r] fp32 gain of the norm, NULL for all ones
 *   rms_eps       added to the mean square (> 0 when rms_norm)
 * Outputs (any may be NULL):
 *   h_out         [T][d_ff] gate pre-activations, fp64
 *   z_out         [T][r] LoPA intermediate V x, fp64 (LoPA only)
 *   active_out    [T][d_ff] 1 if h > t else 0
 *   y_out         [T][d] fp64
 *   macs_out      [T] multiply-adds executed for that token
 * Returns 0, or -1 on a bad argument.
 */
int oracle_ffn_q(int gating, int skip_inactive, int wdt, int T, int d, int d_ff, int r,
                 const float* x, const void* w_gate, const void* lopa_a, const void* lopa_b,
                 const void* w_up, const void* w_down_t, const float* s_gate, const float* s_a,
                 const float* s_b, const float* s_up, const float* s_down, float t, int act, int silu_up,
                 const int32_t* g_idx, const int8_t* g_sign, int rms_norm, const float* rms_gain,
                 float rms_eps, double* h_out, double* z_out, uint8_t* active_out, double* y_out,
                 int64_t* macs_out) {
  if (T < 1 || d < 1 || d_ff < 1 || wdt < 0 || wdt > 3 || !x || !w_up || !w_down_t) return -1;
  if (gating == 0 && !w_gate) return -1;
  if (gating == 1 && (r < 1 || !lopa_a || !lopa_b)) return -1;
  if (gating != 0 && gating != 1) return -1;
  if (wdt >= 2) { /* quantized: every matrix in use has its scales */
    if (!s_up || !s_down || (gating == 0 && !s_gate) || (gating == 1 && (!s_a || !s_b))) return -1;
    if (wdt == 3 && (d % 2 != 0 || (gating == 1 && r % 2 != 0))) return -1;
  }
  if ((act != 0 && act != 1) || (silu_up != 0 && silu_up != 1) || (rms_norm != 0 && rms_norm != 1)) return -1;
  if ((g_idx == NULL) != (g_sign == NULL)) return -1;
  if (gating == 0 && (g_idx || rms_norm)) return -1; /* G and the norm belong to LoPA */
  if (rms_norm && !(rms_eps > 0.0f)) return -1;
  if (g_idx)
    for (int i = 0; i < d_ff; ++i)
      if (g_idx[i] < 0 || g_idx[i] >= d || (g_sign[i] != 1 && g_sign[i] != -1)) return -1;

  const double tt = (double)t;
  int zlen = gating == 1 ? r : 1;

  /* per-call scratch; the oracle is not a hot path */
  double* xv = (double*)malloc(sizeof(double) * (size_t)d);
  double* zv = (double*)malloc(sizeof(double) * (size_t)zlen);
  if (!xv || !zv) {
    free(xv);
    free(zv);
    return -1;
  }

  for (int tok = 0; tok < T; ++tok) {
    int64_t macs = 0;
    for (int j = 0; j < d; ++j) xv[j] = (double)x[(size_t)tok * d + j];

    /* LoPA: the low-rank intermediate z = V x = A x, then the optional RMSNorm */
    if (gating == 1) {
      for (int k = 0; k < r; ++k) zv[k] = row_dot(lopa_a, wdt, s_a, (size_t)k, d, xv, &macs);
      if (z_out)
        for (int k = 0; k < r; ++k) z_out[(size_t)tok * r + k] = zv[k];
      if (rms_norm) {
        double ss = 0.0;
        for (int k = 0; k < r; ++k) ss += zv[k] * zv[k];
        const double inv = 1.0 / sqrt(ss / (double)r + (double)rms_eps);
        for (int k = 0; k < r; ++k) zv[k] = zv[k] * inv * (rms_gain ? (double)rms_gain[k] : 1.0);
      }
    }

    double* y = y_out ? y_out + (size_t)tok * d : NULL;
    if (y)
      for (int j = 0; j < d; ++j) y[j] = 0.0;

    for (int i = 0; i < d_ff; ++i) {
      /* gate pre-activation, computed for every neuron */
      double h = gating == 0 ? row_dot(w_gate, wdt, s_gate, (size_t)i, d, xv, &macs)
                             : row_dot(lopa_b, wdt, s_b, (size_t)i, r, zv, &macs);
      if (g_idx) h += (double)g_sign[i] * xv[g_idx[i]]; /* (G x)_i */
      int active = h > tt; /* strict: A(h) is 0 at h == t for both activations; NaN is inactive */
      if (h_out) h_out[(size_t)tok * d_ff + i] = h;
      if (active_out) active_out[(size_t)tok * d_ff + i] = (uint8_t)active;
      if (skip_inactive && !active) continue;

      double u = active ? h - tt : 0.0;
      double a = act == 1 ? u * logistic(u) : u;              /* A(W1 x)_i */
      double v = row_dot(w_up, wdt, s_up, (size_t)i, d, xv, &macs); /* (W3 x)_i */
      if (silu_up) v = v * logistic(v);
      double zi = a * v;
      if (skip_inactive && zi == 0.0) continue; /* s_gated: column i of W2 is not needed */
      /* y += zi * (column i of W2) = zi * w_down_t[i][:] */
      for (int j = 0; j < d; ++j) {
        double wd = weight_at(w_down_t, wdt, s_down, (size_t)i, (size_t)i * d + (size_t)j);
        if (y) y[j] += zi * wd;
      }
      macs += d;
    }
    if (macs_out) macs_out[tok] = macs;
  }
  free(xv);
  free(zv);
  return 0;
}

/* oracle_ffn_q for fp32 / bf16 weights (no scales) */
int oracle_ffn_ex(int gating, int skip_inactive, int wdt, int T, int d, int d_ff, int r,
                  const float* x, const void* w_gate, const void* lopa_a, const void* lopa_b,
                  const void* w_up, const void* w_down_t, float t, int act, int silu_up,
                  const int32_t* g_idx, const int8_t* g_sign, int rms_norm, const float* rms_gain,
                  float rms_eps, double* h_out, double* z_out, uint8_t* active_out, double* y_out,
                  int64_t* macs_out) {
  if (wdt != 0 && wdt != 1) return -1;
  return oracle_ffn_q(gating, skip_inactive, wdt, T, d, d_ff, r, x, w_gate, lopa_a, lopa_b, w_up, w_down_t, NULL,
                      NULL, NULL, NULL, NULL, t, act, silu_up, g_idx, g_sign, rms_norm, rms_gain, rms_eps, h_out,
                      z_out, active_out, y_out, macs_out);
}

/* oracle_ffn_ex with the default form: shifted ReLU, no activation on W3, G = 0, no norm */
int oracle_ffn(int gating, int skip_inactive, int wdt, int T, int d, int d_ff, int r,
               const float* x, const void* w_gate, const void* lopa_a, const void* lopa_b,
               const void* w_up, const void* w_down_t, float t,
               double* h_out, double* z_out, uint8_t* active_out, double* y_out, int64_t* macs_out) {
  return oracle_ffn_ex(gating, skip_inactive, wdt, T, d, d_ff, r, x, w_gate, lopa_a, lopa_b, w_up, w_down_t, t,
                       0, 0, NULL, NULL, 0, NULL, 0.0f, h_out, z_out, active_out, y_out, macs_out);
}

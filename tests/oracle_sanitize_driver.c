/*
 * Drives the reference oracle (oracle/ffn_oracle.c) under AddressSanitizer and
 * UndefinedBehaviorSanitizer: every gating, weight format, form and path on small odd
 * shapes, plus the argument checks.  Built and run by tests/test_oracle_sanitized.py;
 * exits non-zero on a sanitizer report (the build aborts on the first one) or on an
 * unexpected return code.  Inputs come from a fixed linear congruential generator:
 * the oracle's arithmetic is not in question here, only its memory and integer safety.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_ffn_q(int gating, int skip_inactive, int wdt, int T, int d, int d_ff, int r, const float* x,
                 const void* w_gate, const void* lopa_a, const void* lopa_b, const void* w_up, const void* w_down_t,
                 const float* s_gate, const float* s_a, const float* s_b, const float* s_up, const float* s_down,
                 float t, int act, int silu_up, const int32_t* g_idx, const int8_t* g_sign, int rms_norm,
                 const float* rms_gain, float rms_eps, double* h_out, double* z_out, uint8_t* active_out,
                 double* y_out, int64_t* macs_out);

static uint32_t g_state = 12345u;
static uint32_t next_u32(void) {
  g_state = g_state * 1664525u + 1013904223u;
  return g_state;
}
static float next_unit(void) { return (float)(next_u32() >> 8) / 16777216.0f - 0.5f; } /* [-0.5, 0.5) */

/* a weight matrix of `rows` x `cols` logical elements in format wdt, in its own allocation of
   exactly the stored size, so that a read past it is reported */
static void* make_weights(int wdt, int rows, int cols) {
  size_t n = (size_t)rows * (size_t)cols;
  if (wdt == 0) {
    float* w = malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) w[i] = next_unit();
    return w;
  }
  if (wdt == 1) {
    uint16_t* w = malloc(n * sizeof(uint16_t));
    for (size_t i = 0; i < n; ++i) w[i] = (uint16_t)(0x3C00u + (next_u32() >> 24)) ^ (uint16_t)((next_u32() & 1u) << 15);
    return w;
  }
  if (wdt == 2) {
    int8_t* w = malloc(n);
    for (size_t i = 0; i < n; ++i) w[i] = (int8_t)(next_u32() >> 24);
    return w;
  }
  uint8_t* w = malloc(n / 2); /* two int4 codes a byte */
  for (size_t i = 0; i < n / 2; ++i) w[i] = (uint8_t)(next_u32() >> 24);
  return w;
}

static float* make_scales(int n) {
  float* s = malloc((size_t)n * sizeof(float));
  for (int i = 0; i < n; ++i) s[i] = 0.01f + 0.001f * (float)(next_u32() % 100u);
  return s;
}

static int failures = 0;

static void run_case(int gating, int skip, int wdt, int T, int d, int d_ff, int r, int full) {
  float* x = malloc((size_t)T * d * sizeof(float));
  for (int i = 0; i < T * d; ++i) x[i] = 3.0f * next_unit();
  void* wg = gating == 0 ? make_weights(wdt, d_ff, d) : NULL;
  void* wa = gating == 1 ? make_weights(wdt, r, d) : NULL;
  void* wb = gating == 1 ? make_weights(wdt, d_ff, r) : NULL;
  void* wu = make_weights(wdt, d_ff, d);
  void* wd = make_weights(wdt, d_ff, d);
  const int q = wdt >= 2;
  float* sg = q && gating == 0 ? make_scales(d_ff) : NULL;
  float* sa = q && gating == 1 ? make_scales(r) : NULL;
  float* sb = q && gating == 1 ? make_scales(d_ff) : NULL;
  float* su = q ? make_scales(d_ff) : NULL;
  float* sd = q ? make_scales(d_ff) : NULL;
  int32_t* gi = NULL;
  int8_t* gs = NULL;
  float* gain = NULL;
  if (full && gating == 1) {
    gi = malloc((size_t)d_ff * sizeof(int32_t));
    gs = malloc((size_t)d_ff);
    gain = malloc((size_t)r * sizeof(float));
    for (int i = 0; i < d_ff; ++i) {
      gi[i] = (int32_t)(next_u32() % (uint32_t)d);
      gs[i] = (next_u32() & 1u) ? 1 : -1;
    }
    for (int k = 0; k < r; ++k) gain[k] = 1.0f + next_unit();
  }
  double* h = malloc((size_t)T * d_ff * sizeof(double));
  double* z = gating == 1 ? malloc((size_t)T * r * sizeof(double)) : NULL;
  uint8_t* on = malloc((size_t)T * d_ff);
  double* y = malloc((size_t)T * d * sizeof(double));
  int64_t* macs = malloc((size_t)T * sizeof(int64_t));
  const int rc = oracle_ffn_q(gating, skip, wdt, T, d, d_ff, r, x, wg, wa, wb, wu, wd, sg, sa, sb, su, sd, 0.1f, full,
                              full, gi, gs, full && gating == 1, gain, 1e-6f, h, z, on, y, macs);
  if (rc != 0) {
    fprintf(stderr, "case gating=%d skip=%d wdt=%d T=%d d=%d d_ff=%d r=%d full=%d: rc %d\n", gating, skip, wdt, T, d,
            d_ff, r, full, rc);
    ++failures;
  }
  for (int i = 0; i < T * d; ++i)
    if (!isfinite(y[i])) {
      fprintf(stderr, "case gating=%d wdt=%d: non-finite output\n", gating, wdt);
      ++failures;
      break;
    }
  free(x), free(wg), free(wa), free(wb), free(wu), free(wd);
  free(sg), free(sa), free(sb), free(su), free(sd), free(gi), free(gs), free(gain);
  free(h), free(z), free(on), free(y), free(macs);
}

static void expect_reject(int rc, const char* what) {
  if (rc != -1) {
    fprintf(stderr, "bad argument accepted: %s (rc %d)\n", what, rc);
    ++failures;
  }
}

int main(void) {
  for (int gating = 0; gating <= 1; ++gating)
    for (int skip = 0; skip <= 1; ++skip)
      for (int wdt = 0; wdt <= 3; ++wdt)
        for (int full = 0; full <= 1; ++full) {
          if (full && gating == 0) continue; /* G and the norm belong to LoPA */
          run_case(gating, skip, wdt, 3, 10, 13, 6, full);
          run_case(gating, skip, wdt, 1, 2, 1, 2, full);
        }
  /* argument checks: each must return -1 before touching any array */
  float x[4] = {0};
  uint16_t w[64] = {0};
  int32_t bad_col[4] = {0, 0, 9, 0}, col[4] = {0, 1, 2, 3};
  int8_t sign[4] = {1, 1, 1, 1}, bad_sign[4] = {1, 0, 1, 1};
  expect_reject(oracle_ffn_q(0, 1, 1, 0, 4, 4, 0, x, w, 0, 0, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0),
                "T = 0");
  expect_reject(oracle_ffn_q(1, 1, 1, 1, 4, 4, 0, x, 0, w, w, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0),
                "LoPA with r = 0");
  expect_reject(oracle_ffn_q(0, 1, 2, 1, 4, 4, 0, x, w, 0, 0, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0),
                "int8 without scales");
  expect_reject(oracle_ffn_q(1, 1, 1, 1, 4, 4, 2, x, 0, w, w, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, bad_col, sign, 0, 0, 0.f, 0, 0,
                             0, 0, 0),
                "G column out of range");
  expect_reject(oracle_ffn_q(1, 1, 1, 1, 4, 4, 2, x, 0, w, w, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, col, bad_sign, 0, 0, 0.f, 0,
                             0, 0, 0, 0),
                "G sign 0");
  expect_reject(oracle_ffn_q(1, 1, 1, 1, 4, 4, 2, x, 0, w, w, w, w, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 1, 0, 0.f, 0, 0, 0, 0, 0),
                "RMSNorm with eps 0");
  expect_reject(oracle_ffn_q(1, 1, 3, 1, 3, 4, 2, x, 0, w, w, w, w, 0, x, x, x, x, 0.f, 0, 0, 0, 0, 0, 0, 0.f, 0, 0, 0, 0, 0),
                "int4 with odd d");
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("oracle sanitized run: ok\n");
  return 0;
}

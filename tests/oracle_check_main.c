/*
 * Test driver for the CPU oracle built with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_oracle_sanitized.py).
 *
 * One oracle routine per run: argv[1] names it, the remaining arguments are
 * its sizes and scalars, its input arrays arrive on stdin as raw bytes in
 * the order listed below, and its outputs leave on stdout as raw bytes in
 * the order listed.  Every buffer is allocated at its exact size, so any
 * access one element past an array is reported by the sanitizer, and every
 * buffer is freed, so the leak checker covers the oracle's own allocations.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fgq_oracle.h"

static unsigned char* g_in;
static size_t g_in_len, g_in_pos;

static void die(const char* msg) {
  fprintf(stderr, "oracle_check: %s\n", msg);
  exit(2);
}

static void read_stdin(void) {
  size_t cap = 1 << 16;
  g_in = malloc(cap);
  if (!g_in) die("out of memory");
  for (;;) {
    if (g_in_len == cap) {
      cap *= 2;
      unsigned char* p = realloc(g_in, cap);
      if (!p) die("out of memory");
      g_in = p;
    }
    const size_t n = fread(g_in + g_in_len, 1, cap - g_in_len, stdin);
    if (n == 0) break;
    g_in_len += n;
  }
}

/* The next `bytes` of stdin in a buffer of exactly that size. */
static void* take(size_t bytes) {
  if (g_in_pos + bytes > g_in_len) die("input shorter than the arguments imply");
  void* p = malloc(bytes ? bytes : 1);
  if (!p) die("out of memory");
  memcpy(p, g_in + g_in_pos, bytes);
  g_in_pos += bytes;
  return p;
}

static void* zalloc(size_t bytes) {
  void* p = calloc(bytes ? bytes : 1, 1);
  if (!p) die("out of memory");
  return p;
}

static void put(const void* p, size_t bytes) {
  if (fwrite(p, 1, bytes, stdout) != bytes) die("short write");
}

static int64_t arg_i(int argc, char** argv, int i) {
  if (i >= argc) die("missing argument");
  return strtoll(argv[i], NULL, 10);
}

static float arg_f(int argc, char** argv, int i) {
  if (i >= argc) die("missing argument");
  return (float)strtod(argv[i], NULL);
}

static void check(int rc) {
  if (rc != 0) {
    fprintf(stderr, "oracle_check: status %d\n", rc);
    exit(3);
  }
}

/* Convolution geometry shared by the conv routines: B H W C O R S sh sw ph pw. */
struct geom {
  int64_t B, H, W, C, O, R, S, sh, sw, ph, pw, Ho, Wo, M, K;
};

static struct geom read_geom(int argc, char** argv, int i) {
  struct geom g;
  g.B = arg_i(argc, argv, i);
  g.H = arg_i(argc, argv, i + 1);
  g.W = arg_i(argc, argv, i + 2);
  g.C = arg_i(argc, argv, i + 3);
  g.O = arg_i(argc, argv, i + 4);
  g.R = arg_i(argc, argv, i + 5);
  g.S = arg_i(argc, argv, i + 6);
  g.sh = arg_i(argc, argv, i + 7);
  g.sw = arg_i(argc, argv, i + 8);
  g.ph = arg_i(argc, argv, i + 9);
  g.pw = arg_i(argc, argv, i + 10);
  g.Ho = (g.H + 2 * g.ph - g.R) / g.sh + 1;
  g.Wo = (g.W + 2 * g.pw - g.S) / g.sw + 1;
  g.M = g.B * g.Ho * g.Wo;
  g.K = g.R * g.S * g.C;
  return g;
}

static size_t act_bytes(int64_t n, int64_t bits) { return bits == 8 ? (size_t)n : (size_t)(n / 2); }
static size_t code_bytes(int64_t O, int64_t K) { return (size_t)(O * ((K + 3) / 4)); }

int main(int argc, char** argv) {
  if (argc < 2) die("usage: oracle_check <routine> <arguments>");
  read_stdin();
  const char* op = argv[1];
  const int32_t nt = 2;

  if (!strcmp(op, "ternarize")) {
    /* O C R S G method; in w[O*C*R*S]; out t[O*K], alpha[O*K/G], delta[O*K/G] */
    const int64_t O = arg_i(argc, argv, 2), C = arg_i(argc, argv, 3);
    const int32_t R = (int32_t)arg_i(argc, argv, 4), S = (int32_t)arg_i(argc, argv, 5);
    const int32_t G = (int32_t)arg_i(argc, argv, 6), method = (int32_t)arg_i(argc, argv, 7);
    const int64_t K = C * R * S, ng = O * K / G;
    float* w = take(sizeof(float) * O * K);
    int8_t* t = zalloc(O * K);
    float* a = zalloc(sizeof(float) * ng);
    float* d = zalloc(sizeof(float) * ng);
    check(orc_ternarize(w, O, C, R, S, G, method, t, a, d));
    put(t, O * K);
    put(a, sizeof(float) * ng);
    put(d, sizeof(float) * ng);
    free(w); free(t); free(a); free(d);
  } else if (!strcmp(op, "ternarize_asym")) {
    /* O C R S G; in w; out t, alpha, delta_p, delta_n */
    const int64_t O = arg_i(argc, argv, 2), C = arg_i(argc, argv, 3);
    const int32_t R = (int32_t)arg_i(argc, argv, 4), S = (int32_t)arg_i(argc, argv, 5);
    const int32_t G = (int32_t)arg_i(argc, argv, 6);
    const int64_t K = C * R * S, ng = O * K / G;
    float* w = take(sizeof(float) * O * K);
    int8_t* t = zalloc(O * K);
    float* a = zalloc(sizeof(float) * ng);
    float* dp = zalloc(sizeof(float) * ng);
    float* dn = zalloc(sizeof(float) * ng);
    check(orc_ternarize_asym(w, O, C, R, S, G, t, a, dp, dn));
    put(t, O * K);
    put(a, sizeof(float) * ng);
    put(dp, sizeof(float) * ng);
    put(dn, sizeof(float) * ng);
    free(w); free(t); free(a); free(dp); free(dn);
  } else if (!strcmp(op, "ks")) {
    /* n; in w[n]; out d[2] (fp64) */
    const int64_t n = arg_i(argc, argv, 2);
    float* w = take(sizeof(float) * n);
    double* d = zalloc(2 * sizeof(double));
    check(orc_ks_distances(w, n, d));
    put(d, 2 * sizeof(double));
    free(w); free(d);
  } else if (!strcmp(op, "codes")) {
    /* O K; in t[O*K]; out codes, unpacked t */
    const int64_t O = arg_i(argc, argv, 2), K = arg_i(argc, argv, 3);
    int8_t* t = take(O * K);
    uint8_t* c = zalloc(code_bytes(O, K));
    int8_t* t2 = zalloc(O * K);
    orc_pack_codes(t, O, K, c);
    orc_unpack_codes(c, O, K, t2);
    put(c, code_bytes(O, K));
    put(t2, O * K);
    free(t); free(c); free(t2);
  } else if (!strcmp(op, "quantize")) {
    /* n bits has_scale; in x[n] (then scale if has_scale); out q, s */
    const int64_t n = arg_i(argc, argv, 2);
    const int32_t bits = (int32_t)arg_i(argc, argv, 3);
    const int has_scale = (int)arg_i(argc, argv, 4);
    float* x = take(sizeof(float) * n);
    float* sin = has_scale ? take(sizeof(float)) : NULL;
    uint8_t* q = zalloc(act_bytes(n, bits));
    float s = 0.0f;
    check(orc_quantize_act(x, n, bits, sin, q, &s));
    put(q, act_bytes(n, bits));
    put(&s, sizeof s);
    free(x); free(sin); free(q);
  } else if (!strcmp(op, "group_sums") || !strcmp(op, "conv2d") || !strcmp(op, "conv2d_rows") ||
             !strcmp(op, "conv2d_dfp")) {
    /* geometry (11) G bits, then: group_sums row0 nrows | conv2d sx row0 nrows |
     * conv2d_rows sx nrows | conv2d_dfp sx fl row0 nrows.
     * in q, codes, then alpha[O*K/G] (conv2d, conv2d_rows) or A[O*K/G]
     * (conv2d_dfp), then rows[nrows] (conv2d_rows). */
    const struct geom g = read_geom(argc, argv, 2);
    const int32_t G = (int32_t)arg_i(argc, argv, 13), bits = (int32_t)arg_i(argc, argv, 14);
    const int64_t ng = g.O * g.K / G;
    uint8_t* q = take(act_bytes(g.B * g.H * g.W * g.C, bits));
    uint8_t* c = take(code_bytes(g.O, g.K));
    if (!strcmp(op, "group_sums")) {
      const int64_t row0 = arg_i(argc, argv, 15), nrows = arg_i(argc, argv, 16);
      int32_t* P = zalloc(sizeof(int32_t) * nrows * ng);
      check(orc_group_sums_conv(q, bits, g.B, g.H, g.W, g.C, c, g.O, (int32_t)g.R, (int32_t)g.S,
                                (int32_t)g.sh, (int32_t)g.sw, (int32_t)g.ph, (int32_t)g.pw, G, row0,
                                nrows, P));
      put(P, sizeof(int32_t) * nrows * ng);
      free(P);
    } else if (!strcmp(op, "conv2d")) {
      const float sx = arg_f(argc, argv, 15);
      const int64_t row0 = arg_i(argc, argv, 16), nrows = arg_i(argc, argv, 17);
      float* a = take(sizeof(float) * ng);
      float* y = zalloc(sizeof(float) * g.M * g.O);
      check(orc_conv2d(q, bits, sx, g.B, g.H, g.W, g.C, c, a, g.O, (int32_t)g.R, (int32_t)g.S,
                       (int32_t)g.sh, (int32_t)g.sw, (int32_t)g.ph, (int32_t)g.pw, G, row0, nrows,
                       nt, y));
      put(y, sizeof(float) * g.M * g.O);
      free(a); free(y);
    } else if (!strcmp(op, "conv2d_rows")) {
      const float sx = arg_f(argc, argv, 15);
      const int64_t nrows = arg_i(argc, argv, 16);
      float* a = take(sizeof(float) * ng);
      int64_t* rows = take(sizeof(int64_t) * nrows);
      float* y = zalloc(sizeof(float) * nrows * g.O);
      double* mag = zalloc(sizeof(double) * nrows * g.O);
      check(orc_conv2d_rows(q, bits, sx, g.B, g.H, g.W, g.C, c, a, g.O, (int32_t)g.R,
                            (int32_t)g.S, (int32_t)g.sh, (int32_t)g.sw, (int32_t)g.ph,
                            (int32_t)g.pw, G, rows, nrows, nt, y, mag));
      put(y, sizeof(float) * nrows * g.O);
      put(mag, sizeof(double) * nrows * g.O);
      free(a); free(rows); free(y); free(mag);
    } else {
      const float sx = arg_f(argc, argv, 15);
      const int32_t fl = (int32_t)arg_i(argc, argv, 16);
      const int64_t row0 = arg_i(argc, argv, 17), nrows = arg_i(argc, argv, 18);
      int8_t* A = take(ng);
      float* y = zalloc(sizeof(float) * g.M * g.O);
      check(orc_conv2d_dfp(q, bits, sx, g.B, g.H, g.W, g.C, c, A, fl, g.O, (int32_t)g.R,
                           (int32_t)g.S, (int32_t)g.sh, (int32_t)g.sw, (int32_t)g.ph,
                           (int32_t)g.pw, G, row0, nrows, nt, y));
      put(y, sizeof(float) * g.M * g.O);
      free(A); free(y);
    }
    free(q); free(c);
  } else if (!strcmp(op, "gemm") || !strcmp(op, "gemm_dfp")) {
    /* M K O G bits sx (fl for gemm_dfp); in q[M*K*bits/8], codes, alpha or A; out y[M*O] */
    const int64_t M = arg_i(argc, argv, 2), K = arg_i(argc, argv, 3), O = arg_i(argc, argv, 4);
    const int32_t G = (int32_t)arg_i(argc, argv, 5), bits = (int32_t)arg_i(argc, argv, 6);
    const float sx = arg_f(argc, argv, 7);
    const int64_t ng = O * K / G;
    uint8_t* q = take(act_bytes(M * K, bits));
    uint8_t* c = take(code_bytes(O, K));
    float* y = zalloc(sizeof(float) * M * O);
    if (!strcmp(op, "gemm")) {
      float* a = take(sizeof(float) * ng);
      check(orc_gemm(q, bits, sx, M, K, c, a, O, G, nt, y));
      free(a);
    } else {
      const int32_t fl = (int32_t)arg_i(argc, argv, 8);
      int8_t* A = take(ng);
      check(orc_gemm_dfp(q, bits, sx, M, K, c, A, fl, O, G, nt, y));
      free(A);
    }
    put(y, sizeof(float) * M * O);
    free(q); free(c); free(y);
  } else if (!strcmp(op, "dfp_alpha")) {
    /* n bits; in alpha[n]; out A[n], fl */
    const int64_t n = arg_i(argc, argv, 2);
    const int32_t bits = (int32_t)arg_i(argc, argv, 3);
    float* a = take(sizeof(float) * n);
    int8_t* A = zalloc(n);
    int32_t fl = 0;
    check(orc_dfp_alpha(a, n, bits, A, &fl));
    put(A, n);
    put(&fl, sizeof fl);
    free(a); free(A);
  } else if (!strcmp(op, "w8")) {
    /* geometry (11) bits sx row0 nrows; in w[O*C*R*S] (fp32, [O][C][R][S]), q;
     * out W8[O*C*R*S], fl, y[M*O] */
    const struct geom g = read_geom(argc, argv, 2);
    const int32_t bits = (int32_t)arg_i(argc, argv, 13);
    const float sx = arg_f(argc, argv, 14);
    const int64_t row0 = arg_i(argc, argv, 15), nrows = arg_i(argc, argv, 16);
    const int64_t nw = g.O * g.K;
    float* w = take(sizeof(float) * nw);
    uint8_t* q = take(act_bytes(g.B * g.H * g.W * g.C, bits));
    int8_t* W8 = zalloc(nw);
    int32_t fl = 0;
    check(orc_w8_quantize(w, nw, W8, &fl));
    float* y = zalloc(sizeof(float) * g.M * g.O);
    check(orc_conv2d_w8(q, bits, sx, g.B, g.H, g.W, g.C, W8, fl, g.O, (int32_t)g.R, (int32_t)g.S,
                        (int32_t)g.sh, (int32_t)g.sw, (int32_t)g.ph, (int32_t)g.pw, row0, nrows, nt,
                        y));
    put(W8, nw);
    put(&fl, sizeof fl);
    put(y, sizeof(float) * g.M * g.O);
    free(w); free(q); free(W8); free(y);
  } else {
    die("unknown routine");
  }
  if (g_in_pos != g_in_len) die("input longer than the arguments imply");
  free(g_in);
  return 0;
}

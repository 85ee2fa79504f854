/*
 * oracle.c -- plain, slow CPU reference for the FAST block-floating-point (BFP)
 * hot path: FP32 -> BFP conversion and the BFP dot product / GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, import or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no code, header, table or constant with the
 * HIP kernels.
 *
 * Paper: Zhang, McDanel, Kung, "FAST: DNN Training Under Variable Precision
 * Block Floating Point with Stochastic Rounding" (HPCA 2022).
 *
 * Numbers are represented exactly: quantized mantissas as signed integers
 * (sign-magnitude value +-q), shared exponents as the 8-bit FP32 exponent
 * field, products and group sums in 64-bit integers, scaled values and
 * cross-group sums in IEEE double.  Readings of the paper where it is silent
 * (rounding tie rule, saturation, noise width and noise addressing, zero and
 * subnormal handling) are stated next to the code that takes them.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared oracle.c -o liboracle.so -lm
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 counter-based generator.                                    */
/* Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" */
/* (SC'11), section 3 (Philox): a round maps (L0,R0,L1,R1) with two 32x32   */
/* multiplications; the key is bumped by the Weyl constants between rounds. */
/* ------------------------------------------------------------------------ */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u /* golden ratio */
#define PHILOX_W1 0xBB67AE85u /* sqrt(3) - 1 */

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * x2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t y0 = hi1 ^ x1 ^ k0;
    uint32_t y1 = lo1;
    uint32_t y2 = hi0 ^ x3 ^ k1;
    uint32_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/*
 * Noise byte U in [0, 256) for position p of group gid under seed.
 * Reading of the paper's converter (section V-C: 8-bit random streams added to
 * each aligned mantissa) with Philox standing in for the LFSR: one Philox call
 * yields 16 bytes, one per position of a 16-value block of the group.
 *   key     = (seed mod 2^32, seed div 2^32)
 *   counter = (gid mod 2^32, gid div 2^32, p div 16, 0)
 *   U       = byte (p mod 4), little-endian, of output word ((p div 4) mod 4)
 * gid is the flat index of the group in the output exponent array, so the
 * noise is a function of (seed, output element) and not of any launch shape.
 */
uint32_t oracle_noise_byte(uint64_t seed, uint64_t gid, uint32_t p) {
  uint32_t ctr[4] = {(uint32_t)gid, (uint32_t)(gid >> 32), p / 16u, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  return (w[(p / 4u) % 4u] >> (8u * (p % 4u))) & 0xFFu;
}

/*
 * The noise bytes of ngroups consecutive groups gid0, gid0 + 1, ... with g
 * positions each: out[i * g + p] = oracle_noise_byte(seed, gid0 + i, p).
 */
void oracle_noise_bytes(uint64_t seed, uint64_t gid0, int64_t ngroups, int g, uint8_t* out) {
  for (int64_t i = 0; i < ngroups; ++i)
    for (int p = 0; p < g; ++p) out[i * g + p] = (uint8_t)oracle_noise_byte(seed, gid0 + (uint64_t)i, (uint32_t)p);
}

/* ------------------------------------------------------------------------ */
/* FP32 -> BFP conversion of one group (section III-A and the converter of   */
/* section V-C).                                                             */
/* ------------------------------------------------------------------------ */
enum { ORACLE_NEAREST = 0, ORACLE_STOCHASTIC = 1, ORACLE_TRUNCATE = 2 };

/* Biased exponent field of an FP32 value; subnormals flush to zero (their
 * field is already 0).  Reading: the paper does not treat subnormals. */
static int exponent_field(float v) {
  uint32_t b;
  memcpy(&b, &v, 4);
  return (int)((b >> 23) & 0xFFu);
}

/*
 * Quantize g values x[0..g) (element k at x[k*stride]) to a BFP group with an
 * m-bit magnitude per element and one shared exponent.
 *   noise[k] (0..255) is the stochastic-rounding byte of element k; it is read
 *   only in ORACLE_STOCHASTIC mode.
 * Outputs: q[k*qstride] = sign(x_k) * magnitude (an integer in [-(2^m-1), 2^m-1]),
 *          *E = the shared exponent field.
 * Returns 1 if a non-finite input was seen (a precondition violation), else 0.
 */
static int quantize_group_floor(const float* x, int64_t stride, int g, int m, int mode, const uint8_t* noise,
                                int16_t* q, int64_t qstride, uint8_t* E, int emin);

int oracle_quantize_group(const float* x, int64_t stride, int g, int m, int mode, const uint8_t* noise,
                          int16_t* q, int64_t qstride, uint8_t* E) {
  return quantize_group_floor(x, stride, g, m, mode, noise, q, qstride, E, 0);
}

/*
 * The same conversion with the shared exponent raised to at least emin: the
 * packed layout's exponent of section V-D has a few bits above a base shared
 * by the tensor, so a group whose largest exponent lies below the base is
 * converted at the base (its values aligned to the base's, coarser, LSB).
 * With emin = 0 this is oracle_quantize_group.
 */
int oracle_quantize_group_floor(const float* x, int64_t stride, int g, int m, int mode, const uint8_t* noise,
                                int16_t* q, int64_t qstride, uint8_t* E, int emin) {
  return quantize_group_floor(x, stride, g, m, mode, noise, q, qstride, E, emin);
}

static int quantize_group_floor(const float* x, int64_t stride, int g, int m, int mode, const uint8_t* noise,
                                int16_t* q, int64_t qstride, uint8_t* E, int emin) {
  int bad = 0;
  /* (a) the largest exponent in the group becomes the shared exponent (no
   * lower than emin). */
  int emax = emin;
  for (int k = 0; k < g; ++k) {
    int e = exponent_field(x[k * stride]);
    if (e == 255) bad = 1;
    if (e > emax) emax = e;
  }
  *E = (uint8_t)emax;
  /* Reading: the leading bit of the largest magnitude sits in the top bit of
   * the m-bit field, so one unit in the last place is 2^(E-127-(m-1)). */
  const int lsb_exp = emax - 127 - (m - 1);
  const double qmax = ldexp(1.0, m) - 1.0;
  for (int k = 0; k < g; ++k) {
    float v = x[k * stride];
    int e = exponent_field(v);
    /* (b) align: the magnitude expressed in units of the shared LSB.  A power
     * of two scaling, so it is exact in double; it lies in [0, 2^m).
     * Subnormal inputs (field 0) flush to zero. */
    double a = (e == 0) ? 0.0 : ldexp(fabs((double)v), -lsb_exp);
    /* (c) add noise below the LSB.  Stochastic rounding adds an 8-bit random
     * stream (U/256 of an LSB); round-to-nearest adds exactly half an LSB
     * (ties go away from zero); truncation adds nothing. */
    double u = 0.0;
    if (mode == ORACLE_STOCHASTIC) u = (double)noise[k] / 256.0;
    else if (mode == ORACLE_NEAREST) u = 0.5;
    /* (d) truncate the low-order bits to the m-bit field.  a has at most 24
     * significant bits and u is a multiple of 2^-8 below 1, so a + u is exact
     * to well below 2^-44 and floor() sees the exact sum's integer part. */
    double t = floor(a + u);
    /* Reading: a group maximum that rounds up to 2^m saturates at 2^m - 1 so
     * that the shared exponent stays the group's largest exponent. */
    if (t > qmax) t = qmax;
    int mag = (int)t;
    q[k * qstride] = (int16_t)(signbit(v) ? -mag : mag);
  }
  return bad;
}

/*
 * Quantize output rows [r0, r1) of a row-major matrix x[R][C].
 * axis = 1: groups are g consecutive elements of a row; the full output is
 *           q[R][C], E[R][C/g]; group gid = r*(C/g) + j.
 * axis = 0: groups are g consecutive elements of a column; the full output is
 *           laid out along the new last axis, q[C][R], E[C][R/g]; output row r
 *           is column r of x, and gid = r*(R/g) + j.
 * Only output rows r0..r1-1 are written, to q[(r-r0)*len ...] and
 * E[(r-r0)*(len/g) ...]; gid always uses the absolute row r.
 * Returns the number of groups that held a non-finite input.
 */
/*
 * The exponent base of the packed layout (section V-D: a group's exponent in
 * ebits bits): the largest exponent field of the tensor's values minus
 * 2^ebits - 1, and at least 0, so that every group's exponent, raised to at
 * least the base, is the base plus an ebits-bit offset.
 */
int oracle_exponent_base(const float* x, int64_t n, int ebits) {
  int emax = 0;
  for (int64_t i = 0; i < n; ++i) {
    int e = exponent_field(x[i]);
    if (e > emax) emax = e;
  }
  int base = emax - ((1 << ebits) - 1);
  return base > 0 ? base : 0;
}

static int64_t quantize_rows_floor(const float* x, int64_t R, int64_t C, int axis, int g, int m, int mode,
                                   uint64_t seed, int64_t r0, int64_t r1, int16_t* q, uint8_t* E, int emin);

int64_t oracle_quantize(const float* x, int64_t R, int64_t C, int axis, int g, int m, int mode, uint64_t seed,
                        int64_t r0, int64_t r1, int16_t* q, uint8_t* E) {
  return quantize_rows_floor(x, R, C, axis, g, m, mode, seed, r0, r1, q, E, 0);
}

/* oracle_quantize with every shared exponent raised to at least emin. */
int64_t oracle_quantize_floor(const float* x, int64_t R, int64_t C, int axis, int g, int m, int mode, uint64_t seed,
                              int emin, int64_t r0, int64_t r1, int16_t* q, uint8_t* E) {
  return quantize_rows_floor(x, R, C, axis, g, m, mode, seed, r0, r1, q, E, emin);
}

static int64_t quantize_rows_floor(const float* x, int64_t R, int64_t C, int axis, int g, int m, int mode,
                                   uint64_t seed, int64_t r0, int64_t r1, int16_t* q, uint8_t* E, int emin) {
  int64_t bad = 0;
  const int64_t out_len = (axis == 1) ? C : R; /* elements per output row */
  const int64_t ngroups = out_len / g;
  uint8_t noise[256];
  for (int64_t r = r0; r < r1; ++r) {
    for (int64_t j = 0; j < ngroups; ++j) {
      const int64_t gid = r * ngroups + j;
      if (mode == ORACLE_STOCHASTIC)
        for (int k = 0; k < g; ++k) noise[k] = (uint8_t)oracle_noise_byte(seed, (uint64_t)gid, (uint32_t)k);
      const float* src;
      int64_t stride;
      if (axis == 1) {
        src = x + r * C + j * g;
        stride = 1;
      } else {
        src = x + (j * g) * C + r; /* column r, rows j*g .. j*g+g-1 */
        stride = C;
      }
      bad += quantize_group_floor(src, stride, g, m, mode, noise, q + (r - r0) * out_len + j * g, 1,
                                  E + (r - r0) * ngroups + j, emin);
    }
  }
  return bad;
}

/* BFP -> real value: +-q * 2^(E-127-(m-1)), exact in double.  Rows [r0, r1). */
void oracle_dequantize(const int16_t* q, const uint8_t* E, int64_t len, int g, int m, int64_t r0, int64_t r1,
                       double* y) {
  const int64_t ng = len / g;
  for (int64_t r = r0; r < r1; ++r)
    for (int64_t k = 0; k < len; ++k)
      y[r * len + k] = ldexp((double)q[r * len + k], (int)E[r * ng + k / g] - 127 - (m - 1));
}

/* ------------------------------------------------------------------------ */
/* BFP dot product and GEMM (section III-B, fMAC of section V-B).            */
/* ------------------------------------------------------------------------ */

/* Lower a stored magnitude to m_use bits by dropping its low-order bits (the
 * paper discards low-order mantissa chunks when a lower precision is chosen,
 * section V-D).  Truncation toward zero, sign kept. */
static int64_t lower_precision(int v, int m_stored, int m_use) {
  int s = m_stored - m_use;
  int mag = v < 0 ? -v : v;
  mag >>= s;
  return v < 0 ? -(int64_t)mag : (int64_t)mag;
}

/*
 * C = A * B^T for BFP operands with groups of g along K.
 *   A: qa[M][K] (+-magnitude at a_m stored bits), ea[M][K/g]
 *   B: qb[N][K] (+-magnitude at b_m stored bits), eb[N][K/g]
 *   m_a <= a_m, m_b <= b_m: the precisions the product is taken at.
 * For the output rows listed in rows[0..nrows) (all rows if rows == NULL and
 * nrows == M), writes, at position t*N + j:
 *   C[t][j]      = sum over groups G of T_G, where
 *   T_G          = P_G * 2^(ea + eb - 254 - (m_a-1) - (m_b-1)),
 *   P_G          = sum_{k in G} qa'[i][k] * qb'[j][k]   (exact integer: part M
 *                  and part A of the paper's group dot product),
 *   sumabs[t][j] = sum over groups of |T_G|   (for the error bound).
 * T_G is exact in double; the cross-group sum is accumulated in double, error
 * at most (K/g) * 2^-53 * sumabs.
 */
void oracle_gemm(const int16_t* qa, const uint8_t* ea, int a_m, const int16_t* qb, const uint8_t* eb, int b_m,
                 int64_t M, int64_t N, int64_t K, int g, int m_a, int m_b, const int64_t* rows, int64_t nrows,
                 double* C, double* sumabs) {
  (void)M;
  const int64_t ng = K / g;
  for (int64_t t = 0; t < nrows; ++t) {
    const int64_t i = rows ? rows[t] : t;
    for (int64_t j = 0; j < N; ++j) {
      double acc = 0.0, accabs = 0.0;
      for (int64_t G = 0; G < ng; ++G) {
        int64_t P = 0;
        for (int64_t k = G * g; k < (G + 1) * g; ++k)
          P += lower_precision(qa[i * K + k], a_m, m_a) * lower_precision(qb[j * K + k], b_m, m_b);
        const int sc = (int)ea[i * ng + G] + (int)eb[j * ng + G] - 254 - (m_a - 1) - (m_b - 1);
        const double T = ldexp((double)P, sc);
        acc += T;
        accabs += fabs(T);
      }
      C[t * N + j] = acc;
      if (sumabs) sumabs[t * N + j] = accabs;
    }
  }
}

/*
 * Integer group partials P[G][i][j] = sum_{k in G} qa'[i][k] * qb'[j][k] for
 * the output rows in rows[0..nrows) (P laid out [ng][nrows][N]).
 */
void oracle_group_partials(const int16_t* qa, int a_m, const int16_t* qb, int b_m, int64_t N, int64_t K, int g,
                           int m_a, int m_b, const int64_t* rows, int64_t nrows, int64_t* P) {
  const int64_t ng = K / g;
  for (int64_t G = 0; G < ng; ++G)
    for (int64_t t = 0; t < nrows; ++t) {
      const int64_t i = rows ? rows[t] : t;
      for (int64_t j = 0; j < N; ++j) {
        int64_t s = 0;
        for (int64_t k = G * g; k < (G + 1) * g; ++k)
          s += lower_precision(qa[i * K + k], a_m, m_a) * lower_precision(qb[j * K + k], b_m, m_b);
        P[(G * nrows + t) * N + j] = s;
      }
    }
}

/*
 * Relative improvement r(X) of Eq. 2 (section IV-B): sum_n |BFP(X_n,4) -
 * BFP(X_n,2)| / sum_n |BFP(X_n,2)|, given both quantizations of the same
 * tensor (values dequantized by the caller or here from q/E).  Accumulates
 * the numerator and denominator over rows [r0, r1) into num[0], den[0].
 */
void oracle_relative_improvement(const int16_t* q4, const uint8_t* e4, const int16_t* q2, const uint8_t* e2,
                                 int64_t len, int g, int64_t r0, int64_t r1, double* num, double* den) {
  const int64_t ng = len / g;
  double n = 0.0, d = 0.0;
  for (int64_t r = r0; r < r1; ++r)
    for (int64_t k = 0; k < len; ++k) {
      double v4 = ldexp((double)q4[r * len + k], (int)e4[r * ng + k / g] - 127 - 3);
      double v2 = ldexp((double)q2[r * len + k], (int)e2[r * ng + k / g] - 127 - 1);
      n += fabs(v4 - v2);
      d += fabs(v2);
    }
  num[0] += n;
  den[0] += d;
}

/* ------------------------------------------------------------------------ */
/* Adaptive precision (section IV-B: Algorithm 1 and Eqs. 1-2; section V-D).  */
/* ------------------------------------------------------------------------ */

/*
 * The 2-bit mantissa of the adaptive scheme, taken from the stored 4-bit one:
 * the converter keeps 4-bit mantissas as two 2-bit chunks and, when 2 bits
 * are selected, the low chunk is discarded (section V-D).  The shared
 * exponent is unchanged, so BFP(X,2) = sign * (|q4| >> 2) * 2^(E-127-1).
 */
void oracle_drop_low_chunk(const int16_t* q4, int64_t n, int16_t* q2) {
  for (int64_t i = 0; i < n; ++i) {
    const int mag = q4[i] < 0 ? -q4[i] : q4[i];
    q2[i] = (int16_t)(q4[i] < 0 ? -(mag >> 2) : (mag >> 2));
  }
}

/* Eq. 1: the threshold at layer l of L and iteration i of I. */
double oracle_threshold(double alpha, double beta, int64_t i, int64_t I, int64_t l, int64_t L) {
  return alpha - beta * (double)i / (double)I - beta * (double)l / (double)L;
}

/*
 * Algorithm 1's choice for one tensor: 2 bits when the relative improvement
 * r(X) = num / den of 4 over 2 bits is below the threshold, else 4.  An
 * all-zero tensor (den = 0) has no improvement and takes 2 bits.
 */
int oracle_select_mantissa(double num, double den, double eps) {
  const double r = den > 0.0 ? num / den : 0.0;
  return r < eps ? 2 : 4;
}

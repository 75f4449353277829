/*
 * Reference oracle for the CNN forward contraction -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is not part of the product path.  Only the test-suite, the smoke
 * check and the benchmark's CPU-baseline leg load it.  It shares no code,
 * header or constant with the GPU library.
 *
 * What it computes (paper, Sec. 1, the CNN equation, and Listing 1 "CNN
 * loops", with the strides of that equation restored):
 *
 *   Out[b][k][w][h] = sum_{c<Nc} sum_{r<Nr} sum_{s<Ns}
 *                       In[b][c][sw*w + r][sh*h + s] * Ker[k][c][r][s]
 *
 * for b<Nb, k<Nk, w<Nw, h<Nh.  The convolution is "valid": In has spatial
 * extent Nx = sw*(Nw-1)+Nr by Ny = sh*(Nh-1)+Ns.  Arrays are dense,
 * row-major in the index order written above (last index fastest).  The
 * listing accumulates with "+="; the result here starts from zero, which is
 * the same as running the listing on a zeroed Out.
 *
 * Arithmetic is IEEE fp64.  Callers hand in the exact stored input values
 * already widened to double (fp32 and bf16 widen exactly).
 *
 * Besides Out the oracle can also return Abs[b][k][w][h] =
 * sum |In * Ker| over the same (c, r, s), which bounds the rounding error
 * of any summation order and is used to condition error metrics.
 *
 * Loop order follows Listing 1: b, h, w, k, then c, r, s innermost.
 * Threads (OpenMP) split the independent (b, h) iterations; every output is
 * still summed by one thread in the listing's c, r, s order.
 */
#include <stddef.h>
#include <stdint.h>
#include <math.h>

#ifdef _OPENMP
#include <omp.h>
#endif

typedef long long i64;

/* Validate the problem sizes; return 0 when usable, -1 otherwise. */
static int oracle_check(i64 Nb, i64 Nc, i64 Nk, i64 Nw, i64 Nh, i64 Nr, i64 Ns,
                        i64 sw, i64 sh) {
  if (Nb < 1 || Nc < 1 || Nk < 1 || Nw < 1 || Nh < 1 || Nr < 1 || Ns < 1)
    return -1;
  if (sw < 1 || sh < 1) return -1;
  return 0;
}

/* One output point, summed over (c, r, s) in Listing 1 order. */
static void oracle_point(const double* In, const double* Ker,
                         i64 Nc, i64 Nr, i64 Ns, i64 Nx, i64 Ny,
                         i64 sw, i64 sh, i64 b, i64 k, i64 w, i64 h,
                         double* out, double* abs_out) {
  double acc = 0.0, aacc = 0.0;
  for (i64 c = 0; c < Nc; ++c) {
    const double* in_plane = In + (b * Nc + c) * Nx * Ny;
    const double* ker_cs = Ker + (k * Nc + c) * Nr * Ns;
    for (i64 r = 0; r < Nr; ++r) {
      for (i64 s = 0; s < Ns; ++s) {
        double p = in_plane[(sw * w + r) * Ny + (sh * h + s)] * ker_cs[r * Ns + s];
        acc += p;
        aacc += fabs(p);
      }
    }
  }
  *out = acc;
  if (abs_out) *abs_out = aacc;
}

/*
 * Full forward result.  Out (and Abs if non-NULL) have Nb*Nk*Nw*Nh doubles.
 * Returns 0 on success, -1 on bad sizes.
 */
int cnn_oracle_fwd(const double* In, const double* Ker, double* Out, double* Abs,
                   i64 Nb, i64 Nc, i64 Nk, i64 Nw, i64 Nh, i64 Nr, i64 Ns,
                   i64 sw, i64 sh) {
  if (oracle_check(Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)) return -1;
  const i64 Nx = sw * (Nw - 1) + Nr;
  const i64 Ny = sh * (Nh - 1) + Ns;
#pragma omp parallel for collapse(2) schedule(static)
  for (i64 b = 0; b < Nb; ++b) {
    for (i64 h = 0; h < Nh; ++h) {
      for (i64 w = 0; w < Nw; ++w) {
        for (i64 k = 0; k < Nk; ++k) {
          i64 o = ((b * Nk + k) * Nw + w) * Nh + h;
          oracle_point(In, Ker, Nc, Nr, Ns, Nx, Ny, sw, sh, b, k, w, h,
                       &Out[o], Abs ? &Abs[o] : NULL);
        }
      }
    }
  }
  return 0;
}

/*
 * Selected output points.  idx holds n quadruples (b, k, w, h); Out[i] (and
 * Abs[i] if non-NULL) receive the value at the i-th quadruple.  Returns 0 on
 * success, -1 on bad sizes, -2 if an index is out of range.
 */
int cnn_oracle_points(const double* In, const double* Ker, const i64* idx, i64 n,
                      double* Out, double* Abs,
                      i64 Nb, i64 Nc, i64 Nk, i64 Nw, i64 Nh, i64 Nr, i64 Ns,
                      i64 sw, i64 sh) {
  if (oracle_check(Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)) return -1;
  const i64 Nx = sw * (Nw - 1) + Nr;
  const i64 Ny = sh * (Nh - 1) + Ns;
  for (i64 i = 0; i < n; ++i) {
    i64 b = idx[4 * i], k = idx[4 * i + 1], w = idx[4 * i + 2], h = idx[4 * i + 3];
    if (b < 0 || b >= Nb || k < 0 || k >= Nk || w < 0 || w >= Nw || h < 0 || h >= Nh)
      return -2;
  }
#pragma omp parallel for schedule(static)
  for (i64 i = 0; i < n; ++i) {
    oracle_point(In, Ker, Nc, Nr, Ns, Nx, Ny, sw, sh,
                 idx[4 * i], idx[4 * i + 1], idx[4 * i + 2], idx[4 * i + 3],
                 &Out[i], Abs ? &Abs[i] : NULL);
  }
  return 0;
}

/* Number of OpenMP threads the oracle will use (1 without OpenMP). */
int cnn_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Sets the OpenMP thread count of later calls (n >= 1); returns the count
 * used before.  Timing only: the result of every call is independent of it. */
int cnn_oracle_set_threads(int n) {
#ifdef _OPENMP
  const int was = omp_get_max_threads();
  if (n >= 1) omp_set_num_threads(n);
  return was;
#else
  (void)n;
  return 1;
#endif
}

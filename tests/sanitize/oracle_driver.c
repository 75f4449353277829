/*
 * The fp64 oracle (oracle/conv_oracle.c) under AddressSanitizer and
 * UndefinedBehaviorSanitizer, built with gcc by tests/test_sanitizers.py:
 * full results and selected points, with and without the |In*Ker| sums,
 * over pseudo-random small shapes (strides beyond the stencil included),
 * agreement of the two entry points, and their rejection of bad sizes and
 * out-of-range indices.  Prints one line; exits 0 when all held.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef long long i64;
int cnn_oracle_fwd(const double*, const double*, double*, double*, i64, i64, i64, i64, i64, i64,
                   i64, i64, i64);
int cnn_oracle_points(const double*, const double*, const i64*, i64, double*, double*, i64, i64,
                      i64, i64, i64, i64, i64, i64, i64);

static uint64_t rng_state = 12345;

/* splitmix64 (Steele, Lea and Flood, 2014) */
static uint64_t next_u64(void) {
  uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

static i64 pick(i64 lo, i64 hi) { return lo + (i64)(next_u64() % (uint64_t)(hi - lo + 1)); }

int main(void) {
  int bad = 0, runs = 0;
  for (int it = 0; it < 300; ++it) {
    const i64 Nb = pick(1, 3), Nc = pick(1, 6), Nk = pick(1, 6), Nw = pick(1, 9), Nh = pick(1, 9);
    const i64 Nr = pick(1, 5), Ns = pick(1, 5), sw = pick(1, 4), sh = pick(1, 4);
    const i64 Nx = sw * (Nw - 1) + Nr, Ny = sh * (Nh - 1) + Ns;
    const i64 n_in = Nb * Nc * Nx * Ny, n_ker = Nk * Nc * Nr * Ns, n_out = Nb * Nk * Nw * Nh;
    double* In = malloc(sizeof(double) * n_in);
    double* Ker = malloc(sizeof(double) * n_ker);
    double* Out = malloc(sizeof(double) * n_out);
    double* Abs = malloc(sizeof(double) * n_out);
    for (i64 i = 0; i < n_in; ++i) In[i] = (double)pick(-4, 4);
    for (i64 i = 0; i < n_ker; ++i) Ker[i] = (double)pick(-4, 4);
    bad |= cnn_oracle_fwd(In, Ker, Out, (it & 1) ? Abs : NULL, Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh);
    bad |= cnn_oracle_fwd(In, Ker, Out, Abs, Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh);
    const i64 n = 17;
    i64 idx[4 * 17];
    double pt[17], pa[17];
    for (i64 i = 0; i < n; ++i) {
      idx[4 * i] = pick(0, Nb - 1);
      idx[4 * i + 1] = pick(0, Nk - 1);
      idx[4 * i + 2] = pick(0, Nw - 1);
      idx[4 * i + 3] = pick(0, Nh - 1);
    }
    bad |= cnn_oracle_points(In, Ker, idx, n, pt, pa, Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh);
    for (i64 i = 0; i < n; ++i) {
      const i64 o = ((idx[4 * i] * Nk + idx[4 * i + 1]) * Nw + idx[4 * i + 2]) * Nh + idx[4 * i + 3];
      if (pt[i] != Out[o] || pa[i] != Abs[o]) bad = 1;  /* integer data: exact */
    }
    idx[4 * 5 + 2] = Nw;  /* one index out of range */
    if (cnn_oracle_points(In, Ker, idx, n, pt, NULL, Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh) != -2)
      bad = 1;
    if (cnn_oracle_fwd(In, Ker, Out, NULL, Nb, Nc, Nk, Nw, Nh, Nr, Ns, 0, sh) != -1) bad = 1;
    if (cnn_oracle_fwd(In, Ker, Out, NULL, 0, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh) != -1) bad = 1;
    free(In);
    free(Ker);
    free(Out);
    free(Abs);
    ++runs;
  }
  printf("oracle driver: %d shapes, %s\n", runs, bad ? "FAILED" : "ok");
  return bad;
}

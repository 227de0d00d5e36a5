/*
 * Plain C oracle of the compressed se_a descriptor (test infrastructure).
 *
 * Same mathematics as oracle/se_a.py (paper Sec. II): per atom i and valid
 * neighbour j, x = R~_ij[0] selects an interval of the Hermite table of the
 * type pair (type(i), block(j)); g_m and g'_m are the quintic and its
 * derivative at the local offset t; the forward accumulates
 * T_i[m][k] += g_m R~_ij[k] and then D_i[m][n] = sum_k T_i[m][k] T_i[n][k]
 * (n < M'); the backward writes
 * dE/dR~_ij[k] = sum_m dT[m][k] g_m + (k == 0) sum_m g'_m sum_k' dT[m][k'] R~_ij[k'].
 *
 * Scalar loops only, neighbours in ascending slot order, OpenMP over atoms.
 * Build with -O2 -ffp-contract=off so that every product and sum is rounded
 * on its own.  Table layout (oracle's own): coef[off[p] + (l*M + m)*6 + q],
 * q = 0..5 the coefficients of t^q.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
  int nloc, nnei, ntypes, M, M2;
  const int* sel;          /* [ntypes] */
  const double* lo;        /* [ntypes^2] */
  const double* d1;
  const int64_t* L1;
  const double* d2;
  const int64_t* L2;
  const int64_t* off;      /* [ntypes^2] element offset of each pair's table */
  const double* coef;
  const int* atype;        /* [nloc] */
  const int* nlist;        /* [nloc*nnei] */
  const double* em;        /* [nloc*nnei*4] */
} ref_args;

/* interval index, offset and clamp flag for input x of pair p */
static void locate(const ref_args* a, int p, double x, int64_t* l, double* t, int* clamped) {
  double lo = a->lo[p], d1 = a->d1[p], d2 = a->d2[p];
  int64_t L1 = a->L1[p], L2 = a->L2[p];
  double x_up = lo + (double)L1 * d1;
  double x_end = x_up + (double)L2 * d2;
  *clamped = 0;
  if (x < x_up) {
    double q = floor((x - lo) / d1);
    if (q < 0) q = 0;
    if (q > (double)(L1 - 1)) q = (double)(L1 - 1);
    *l = (int64_t)q;
    *t = x - (lo + q * d1);
  } else if (x < x_end) {
    double q = floor((x - x_up) / d2);
    if (q < 0) q = 0;
    if (q > (double)(L2 - 1)) q = (double)(L2 - 1);
    *l = L1 + (int64_t)q;
    *t = x - (x_up + q * d2);
  } else {
    *l = L1 + L2 - 1;
    *t = d2;
    *clamped = 1;
  }
}

static int block_of(const ref_args* a, int j) {
  int acc = 0;
  for (int b = 0; b < a->ntypes; ++b) {
    acc += a->sel[b];
    if (j < acc) return b;
  }
  return a->ntypes - 1;
}

void ref_forward(const ref_args* a, int64_t i0, int64_t i1, double* T, double* D) {
  const int M = a->M, M2 = a->M2, nnei = a->nnei;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = i0; i < i1; ++i) {
    double* Ti = T + (i - i0) * M * 4;
    memset(Ti, 0, sizeof(double) * M * 4);
    for (int j = 0; j < nnei; ++j) {
      if (a->nlist[i * nnei + j] < 0) continue;
      const double* r = a->em + (i * nnei + j) * 4;
      int p = a->atype[i] * a->ntypes + block_of(a, j);
      int64_t l; double t; int cl;
      locate(a, p, r[0], &l, &t, &cl);
      const double* c = a->coef + a->off[p] + l * M * 6;
      for (int m = 0; m < M; ++m) {
        const double* q = c + m * 6;
        double g = ((((q[5] * t + q[4]) * t + q[3]) * t + q[2]) * t + q[1]) * t + q[0];
        for (int k = 0; k < 4; ++k) Ti[m * 4 + k] += g * r[k];
      }
    }
    double* Di = D + (i - i0) * M * M2;
    for (int m = 0; m < M; ++m)
      for (int n = 0; n < M2; ++n) {
        double s = 0.0;
        for (int k = 0; k < 4; ++k) s += Ti[m * 4 + k] * Ti[n * 4 + k];
        Di[m * M2 + n] = s;
      }
  }
}

void ref_backward(const ref_args* a, int64_t i0, int64_t i1, const double* dT, double* dR) {
  const int M = a->M, nnei = a->nnei;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = i0; i < i1; ++i) {
    const double* dTi = dT + (i - i0) * M * 4;
    for (int j = 0; j < nnei; ++j) {
      double* out = dR + ((i - i0) * nnei + j) * 4;
      out[0] = out[1] = out[2] = out[3] = 0.0;
      if (a->nlist[i * nnei + j] < 0) continue;
      const double* r = a->em + (i * nnei + j) * 4;
      int p = a->atype[i] * a->ntypes + block_of(a, j);
      int64_t l; double t; int cl;
      locate(a, p, r[0], &l, &t, &cl);
      const double* c = a->coef + a->off[p] + l * M * 6;
      for (int m = 0; m < M; ++m) {
        const double* q = c + m * 6;
        double g = ((((q[5] * t + q[4]) * t + q[3]) * t + q[2]) * t + q[1]) * t + q[0];
        double gp = cl ? 0.0
                       : (((5.0 * q[5] * t + 4.0 * q[4]) * t + 3.0 * q[3]) * t + 2.0 * q[2]) * t + q[1];
        double w = 0.0;
        for (int k = 0; k < 4; ++k) {
          out[k] += dTi[m * 4 + k] * g;
          w += dTi[m * 4 + k] * r[k];
        }
        out[0] += gp * w;
      }
    }
  }
}

int ref_num_threads(void) {
  int n = 1;
#ifdef _OPENMP
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
#endif
  return n;
}

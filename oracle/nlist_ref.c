/*
 * Plain C oracle of the neighbour list (test infrastructure).
 *
 * Paper Sec. II, the environment matrix: the rows of R~_i are the neighbours
 * j of atom i within the cutoff r_c, grouped by neighbour type (sel_beta rows
 * for type beta), sorted by distance inside each group, and the unused rows
 * are filled with zeros (here: slot index -1).
 *
 * Definition written out by brute force, one atom at a time:
 *   - periodic cubic box of edge `box`, minimum image per component:
 *       d = x_j - x_i,  d = d - box * rint(d / box);
 *   - r2 = dx*dx + dy*dy + dz*dz, each product and sum rounded on its own
 *     (build with -ffp-contract=off), summed in that order;
 *   - j != i is a neighbour when r2 < rc*rc;
 *   - neighbours are ordered by (type, r2, j) ascending; the first sel[beta]
 *     of type beta fill block beta, the rest are dropped and counted.
 * O(n^2) per call, OpenMP over centre atoms.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int type;
  int j;
  double r2;
} nl_cand;

static int cand_less(const nl_cand* a, const nl_cand* b) {
  if (a->type != b->type) return a->type < b->type;
  if (a->r2 != b->r2) return a->r2 < b->r2;
  return a->j < b->j;
}

static int cand_cmp(const void* pa, const void* pb) {
  const nl_cand* a = (const nl_cand*)pa;
  const nl_cand* b = (const nl_cand*)pb;
  if (cand_less(a, b)) return -1;
  if (cand_less(b, a)) return 1;
  return 0;
}

static double min_image(double d, double box) { return d - box * rint(d / box); }

/* Neighbour lists of the atoms `centres[0..ncentre)` (indices into coord);
 * nlist out [ncentre][sum(sel)]; counts out [ncentre][ntypes] = neighbours
 * of each type within rc before truncation.  Returns the number of centres
 * with some type over its sel. */
int ref_nlist(int natoms, const double* coord, const int* atype, int ntypes, const int* sel,
              double box, double rc, int ncentre, const int64_t* centres, int* nlist,
              int* counts) {
  int nnei = 0;
  for (int b = 0; b < ntypes; ++b) nnei += sel[b];
  const double rc2 = rc * rc;
  int over = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(+ : over)
  for (int64_t c = 0; c < ncentre; ++c) {
    const int64_t i = centres[c];
    nl_cand* buf = (nl_cand*)malloc(sizeof(nl_cand) * (size_t)(natoms > 0 ? natoms : 1));
    int n = 0;
    for (int j = 0; j < natoms; ++j) {
      if (j == i) continue;
      const double dx = min_image(coord[3 * j] - coord[3 * i], box);
      const double dy = min_image(coord[3 * j + 1] - coord[3 * i + 1], box);
      const double dz = min_image(coord[3 * j + 2] - coord[3 * i + 2], box);
      const double r2 = dx * dx + dy * dy + dz * dz;
      if (r2 < rc2) {
        buf[n].type = atype[j];
        buf[n].j = j;
        buf[n].r2 = r2;
        ++n;
      }
    }
    qsort(buf, (size_t)n, sizeof(nl_cand), cand_cmp);
    int* row = nlist + c * nnei;
    for (int s = 0; s < nnei; ++s) row[s] = -1;
    int* cnt = counts + c * ntypes;
    for (int b = 0; b < ntypes; ++b) cnt[b] = 0;
    int trunc = 0;
    for (int e = 0; e < n; ++e) {
      const int b = buf[e].type;
      if (b < 0 || b >= ntypes) continue;
      int start = 0;
      for (int q = 0; q < b; ++q) start += sel[q];
      if (cnt[b] < sel[b])
        row[start + cnt[b]] = buf[e].j;
      else
        trunc = 1;
      ++cnt[b];
    }
    over += trunc;
    free(buf);
  }
  return over;
}

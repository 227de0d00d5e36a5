/*
 * dpc.h -- C ABI of the compressed se_a descriptor library (libdpc.so).
 *
 * DP Compress (Lu et al., arXiv:2107.02103), Sec. II: the embedding net
 * G(s^) of the Deep Potential se_a descriptor is replaced by a table of
 * piecewise fifth-order Hermite polynomials, and the product
 * S_i = G_i^T R~_i (here called T_i, M1 x 4) is evaluated by one fused kernel
 * that never materialises G and skips padded neighbours; then
 * D_i = T_i (T_i<)^T (M1 x M2) with T_i< the first M2 rows of T_i.  The
 * backward kernel maps dE/dT_i to dE/dR~_ij through the polynomial and its
 * derivative, which is what forces need.
 *
 * Conventions
 *  - All arrays are row-major and contiguous; sizes are element counts.
 *  - "device" pointers are HIP device memory on the current device; "host"
 *    pointers are ordinary host memory.  The library never allocates device
 *    memory and keeps no global state: every buffer is owned by the caller.
 *  - Kernels are enqueued on the given stream (a hipStream_t passed as
 *    void*, NULL = the null stream) and the calls return without
 *    synchronising.  Faults inside a kernel surface at the caller's next
 *    synchronisation.
 *  - Every argument is validated on the host before anything is launched;
 *    on error nothing is launched and nothing is written.
 *  - Return value: DPC_OK (0) or a negative DPC_E* code; dpc_strerror()
 *    describes it.
 */
#ifndef DPC_H
#define DPC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DPC_OK 0
#define DPC_EINVAL -1   /* null pointer, bad size/shape, bad dtype, sel/nnei mismatch */
#define DPC_ERANGE -2   /* bad table parameters: stride <= 0, L1 or L2 < 1, non-finite lo */
#define DPC_EHIP -3     /* HIP runtime or launch error */
#define DPC_ENOTSUP -4  /* supported but not implemented sizes (M1 > 256, ntypes > 8) */
#define DPC_EOVERFLOW -5 /* a neighbour list had more atoms of some type within r_c than sel */

#define DPC_MAX_TYPES 8
#define DPC_MAX_M1 256

/* Arithmetic of the kernels.
 *  DPC_F64        float64 table, R~, dE/dT, T, D and dE/dR~.
 *  DPC_F32        float32 table, R~, dE/dT, T, D and dE/dR~, float32 arithmetic.
 *  DPC_F32_ACC64  float32 table, R~ and dE/dT; in the forward the polynomial
 *                 is evaluated in float32, T and D accumulated and stored in
 *                 float64; the backward (m1 <= 128) converts its float32
 *                 inputs to float64 and runs like DPC_F64, dE/dR~ in float64.  */
typedef enum { DPC_F64 = 0, DPC_F32 = 1, DPC_F32_ACC64 = 2 } dpc_dtype;

/* Tabulation range of one embedding net (one ordered type pair).
 * Paper Sec. II: the input s^ is tabulated on [s^(r_c), s^(r_l)] with an
 * equal step; here the main range [lo, x_up], x_up = lo + L1*d1, uses step d1
 * and an extrapolation band [x_up, x_end], x_end = x_up + L2*d2, uses d2.
 * Interval l < L1 covers [lo + l*d1, lo + (l+1)*d1); interval L1 + l covers
 * [x_up + l*d2, x_up + (l+1)*d2).  Inputs below lo use interval 0 (t < 0);
 * inputs at or beyond x_end take the value at x_end and zero derivative.
 * `offset` is the element offset of this pair's coefficients inside the
 * coefficient buffer; dpc_table_layout() fills it.                          */
typedef struct {
  double lo;
  double d1;
  double d2;
  int64_t L1;
  int64_t L2;
  int64_t offset;
} dpc_range;

/* Embedding net of one type pair (host memory, read only).
 * widths[0] must be 1; layer k maps widths[k] -> widths[k+1] with
 * y_{k+1} = tanh(y_k W_k + b_k) (+ [y_k, y_k] when widths[k+1] = 2 widths[k],
 * + y_k when widths[k+1] = widths[k]).  W[k] is [widths[k]][widths[k+1]].  */
typedef struct {
  int n_layers;
  const int* widths;         /* [n_layers + 1] */
  const double* const* W;    /* [n_layers] */
  const double* const* b;    /* [n_layers] */
} dpc_net;

/* Human-readable text of a status code (static storage). */
const char* dpc_strerror(int status);

/* Text of the HIP error behind the calling thread's last DPC_EHIP status
 * ("no error" if there was none). */
const char* dpc_last_hip_error(void);

/* Library version as 10000*major + 100*minor + patch. */
int dpc_version(void);

/* Coefficient layout for `npair` type pairs of width m1.
 * In:  ranges[p].{lo,d1,d2,L1,L2}.  Out: ranges[p].offset (elements) and
 * *total_bytes, the size of the coefficient buffer for `dtype` (DPC_F32 and
 * DPC_F32_ACC64 store float32 coefficients).  The layout of one pair is
 * [L1 + L2][3][DPC_TABLE_LD(m1)][2]: interval l holds 6 * ld elements, and
 * the coefficient of t^q of channel m, t = x - (left node of l), is element
 * DPC_TABLE_AT(ld, q, m) of it, so the coefficients of t^(2j) and t^(2j+1)
 * of one channel are adjacent (one 16-byte float64 load brings both).
 * Channels are padded with zeros to a multiple of 4 so that the kernels can
 * use 16-byte loads without leaving the buffer.                             */
#define DPC_TABLE_LD(m1) (((m1) + 3) / 4 * 4)
#define DPC_TABLE_AT(ld, q, m) (((q) >> 1) * 2 * (ld) + 2 * (m) + ((q) & 1))
int dpc_table_layout(int npair, int m1, dpc_range* ranges, dpc_dtype dtype,
                     size_t* total_bytes);

/* Paper Sec. II, Eqs. for the constraints y, y', y'' at both nodes of each
 * interval and the closed forms for a..f: tabulate `net` (m1 = last width)
 * over `range` and write its (L1 + L2) * 6 * DPC_TABLE_LD(m1) coefficients to `host_out`
 * (host memory, float64 or float32 per `dtype`).  The first and second
 * derivatives of the net are computed in forward mode in float64.          */
int dpc_build_table(const dpc_net* net, const dpc_range* range, dpc_dtype dtype,
                    void* host_out);

/* Forward (paper Sec. II, the fused tabulate-and-contract kernel and D):
 *   T_i[m][k] = sum over valid j of g_m^{a_i b_j}(R~_ij[0]) * R~_ij[k]
 *   D_i[m][n] = sum_k T_i[m][k] * T_i[n][k],  n < m2
 * Geometry: neighbour slot j of atom i belongs to block b_j (the first sel[0]
 * slots are block 0, the next sel[1] block 1, ...), nnei = sum(sel); its
 * table is pair a_i*ntypes + b_j with a_i = atype[i].  nlist[i][j] < 0 marks
 * padding, which is skipped (it contributes exactly zero).
 *   stream   hipStream_t as void*
 *   sel      host [ntypes], ntypes <= DPC_MAX_TYPES
 *   ranges   host [ntypes*ntypes], offsets from dpc_table_layout()
 *   coeff    device, the concatenated tables (float64 or float32 per dtype)
 *   atype    device int32 [nloc], values in [0, ntypes); an atom with another
 *            value gets NaN outputs (nothing is read out of bounds)
 *   nlist    device int32 [nloc][nnei]
 *   em       device R~ [nloc][nnei][4] (float64 for DPC_F64, else float32),
 *            16-byte aligned (rows are read 16 bytes at a time)
 *   T        device out [nloc][m1][4]   (float32 only for DPC_F32)
 *   D        device out [nloc][m1][m2]  (float32 only for DPC_F32)
 * Requires 1 <= m1 <= DPC_MAX_M1, 1 <= m2 <= m1.  nloc = 0 is a no-op.      */
int dpc_se_a_tab_fwd(void* stream, dpc_dtype dtype, int nloc, int ntypes, const int* sel,
                     int m1, int m2, const dpc_range* ranges, const void* coeff,
                     const int* atype, const int* nlist, const void* em,
                     void* T, void* D);

/* Backward of T (forces need dE/dR~, paper Sec. II):
 *   dE/dR~_ij[k] = sum_m dE/dT_i[m][k] g_m(x) + (k == 0) sum_m g'_m(x) w_m,
 *   w_m = sum_k' dE/dT_i[m][k'] R~_ij[k'],  x = R~_ij[0],
 * for valid j; padded rows are written as 0.  For DPC_F64 and DPC_F32_ACC64
 * with m1 <= 128 the channel sums are formed per (interval, atom) pair on the
 * matrix cores in float64, as
 * P[k][q] = sum_m dE/dT_i[m][k] C[m][q] followed by a polynomial in t per
 * neighbour: the same sums in another order of rounding.
 *   dE_dT    device [nloc][m1][4] (float64 for DPC_F64, else float32)
 *   dE_dem   device out [nloc][nnei][4] (float32 only for DPC_F32), 16-byte aligned
 * Other arguments as dpc_se_a_tab_fwd.                                      */
int dpc_se_a_tab_bwd(void* stream, dpc_dtype dtype, int nloc, int ntypes, const int* sel,
                     int m1, const dpc_range* ranges, const void* coeff,
                     const int* atype, const int* nlist, const void* em,
                     const void* dE_dT, void* dE_dem);

/* The backward from dE/dD: dpc_descriptor_bwd fused into dpc_se_a_tab_bwd.
 * The matrix-core backward forms dE/dT of its atoms itself, in a prologue on
 * the matrix cores,
 * from the forward's T and dE/dD (paper Sec. II: D_i = T_i (T_i<)^T), so dE/dT
 * is never stored:
 *   dE/dT_i[m][k] = sum_{n<m2} dE/dD_i[m][n] T_i[n][k] + (m < m2) sum_{m'} dE/dD_i[m'][m] T_i[m'][k],
 * then dE/dR~ as dpc_se_a_tab_bwd.  The result equals the two calls up to the
 * order of rounding.
 *   T       device float64 [nloc][m1][4] (the forward's T), 16-byte aligned
 *   dE_dD   device float64 [nloc][m1][m2], 16-byte aligned
 *   dE_dem  device out float64 [nloc][nnei][4], 16-byte aligned
 * Requires DPC_F64, m1 <= 128 and an even m2 <= 16 (DPC_ENOTSUP otherwise:
 * use the two calls).  Other arguments as dpc_se_a_tab_bwd.                 */
int dpc_se_a_tab_bwd_from_dD(void* stream, dpc_dtype dtype, int nloc, int ntypes, const int* sel,
                             int m1, int m2, const dpc_range* ranges, const void* coeff,
                             const int* atype, const int* nlist, const void* em, const void* T,
                             const void* dE_dD, void* dE_dem);

/* Backward of the descriptor (paper Sec. II: D_i = T_i (T_i<)^T, T_i< the
 * first m2 rows of T_i, i.e. D_i[m][n] = sum_k T_i[m][k] T_i[n][k], n < m2):
 *   dE/dT_i[m][k] = sum_{n<m2} dE/dD_i[m][n] T_i[n][k]
 *                 + (m < m2) sum_{m'} dE/dD_i[m'][m] T_i[m'][k].
 * Its output is the dE_dT input of dpc_se_a_tab_bwd, so that a caller holding
 * dE/dD (from the fitting net) and the forward's T gets dE/dR~ in two calls.
 *   T        device [nloc][m1][4], the forward's T (float64, or float32 for DPC_F32)
 *   dE_dD    device [nloc][m1][m2], same type as T
 *   dE_dT    device out [nloc][m1][4]: float64 for DPC_F64, float32 otherwise
 *            (the type dpc_se_a_tab_bwd takes); must not overlap the inputs
 * Arithmetic is float64 except for DPC_F32.  Requires 1 <= m2 <= m1 <=
 * DPC_MAX_M1 and (4 m1 + m1 (m2 + 1)) elements of the arithmetic type within
 * 64 KiB (DPC_ENOTSUP otherwise; m2 = 16 allows every m1).  nloc = 0 is a
 * no-op.  Errors and ownership as the calls above.                          */
int dpc_descriptor_bwd(void* stream, dpc_dtype dtype, int nloc, int m1, int m2,
                       const void* T, const void* dE_dD, void* dE_dT);

/* Environment matrix R~ from positions (paper Sec. II, Eq. (1) and the
 * normalisation after it).  For slot s of atom i with j = nlist[i][s] >= 0:
 * r_ij = r_j - r_i as the minimum image in a cubic periodic box of edge `box`,
 * r = |r_ij|, s(r) = 1/r (r < rcs), (1/r)[u^3(-6u^2+15u-10)+1] (rcs <= r < rc,
 * u = (r - rcs)/(rc - rcs)), 0 (r >= rc), and the row is
 *   ((s - mean[t]) / sigma[t], s x / sigma_all[t], s y / sigma_all[t], s z / sigma_all[t]),
 * t = atype[i]; padding rows (nlist < 0) are zero.
 *   box, rc, rcs  require 0 <= rcs < rc and box > 2 rc (else DPC_ERANGE)
 *   mean, sigma, sigma_all  host [ntypes], sigma and sigma_all > 0
 *   coord    device float64 [nloc][3]
 *   atype    device int32 [nloc]; nlist device int32 [nloc][nnei], entries < nloc
 *            (a row with an out-of-range type or neighbour index becomes NaN)
 *   em       device out [nloc][nnei][4]: float64 for DPC_F64, float32 otherwise
 *            (the em input of dpc_se_a_tab_fwd / _bwd in that mode)
 * Arithmetic is float64.  nloc = 0 is a no-op.                              */
int dpc_env_mat_a(void* stream, dpc_dtype dtype, int nloc, int ntypes, int nnei, double box,
                  double rc, double rcs, const double* mean, const double* sigma,
                  const double* sigma_all, const double* coord, const int* atype,
                  const int* nlist, void* em);

/* Reverse slots of a neighbour list, for dpc_force_a: rev[i][s] = the slot of
 * i in the list of j = nlist[i][s], searched in the sel block of i's type
 * (sel as in dpc_se_a_tab_fwd), or -1 if i is not there (and for padding);
 * if j's block holds i more than once, one of those slots.  In lists sorted
 * by distance within each block i sits near j's rank in i's list, where the
 * search looks first; other orders are scanned, with the same result.
 * Build it once per neighbour list.
 *   coord, box  as for the other calls (validated; the search reads only the
 *               lists and atype)
 *   rev   device out int32 [nloc][nnei]                                      */
int dpc_nlist_reverse(void* stream, int nloc, int ntypes, const int* sel, double box,
                      const double* coord, const int* atype, const int* nlist, int* rev);

/* Bytes of device workspace dpc_nlist_build needs for nloc atoms in a cubic
 * box of edge `box` with cutoff rc (the cell list: per-cell counters and
 * offsets, and the atoms in cell order, 32 bytes each); 0 for bad sizes.   */
size_t dpc_nlist_workspace_bytes(int nloc, double box, double rc);

/* Neighbour list (paper Sec. II, the environment matrix: the neighbours of
 * atom i within r_c, grouped by neighbour type into sel[beta] rows for type
 * beta, sorted by distance inside a group, the unused rows empty):
 *   - periodic cubic box of edge `box`, minimum image per component
 *     d = x_j - x_i - box * rint((x_j - x_i) / box);
 *   - r2 = dx*dx + dy*dy + dz*dz, each operation rounded on its own;
 *   - j != i is a neighbour when r2 < rc*rc (and 0 <= atype[j] < ntypes);
 *   - nlist[i][blk(beta) + k] = the k-th neighbour of type beta in the order
 *     (r2, j) ascending, for k < sel[beta]; the remaining slots hold -1.
 * The result does not depend on the order of the atoms inside the cell list
 * (the order is total), so it is reproducible bitwise.
 *   nloc         at most 2^28 (else DPC_ENOTSUP)
 *   box, rc      require rc > 0 and box > 2 rc (else DPC_ERANGE)
 *   sel          host [ntypes], ntypes <= DPC_MAX_TYPES
 *   coord        device float64 [nloc][3] (any real values: positions are
 *                wrapped into the box for the cell list only)
 *   atype        device int32 [nloc]
 *   workspace    device, 256-byte aligned, >= dpc_nlist_workspace_bytes()
 *   nlist        device out int32 [nloc][sum(sel)] (the nlist input of the
 *                calls above)
 *   status_host  host int [2] or NULL.  With NULL the call is asynchronous
 *                like the others; the two status counters it leaves in the
 *                first 8 bytes of the workspace are the numbers of atoms
 *                whose list was truncated (some type had more than sel
 *                neighbours: its nearest sel are kept) and of atoms with
 *                more than 1024 atoms within rc (their list is incomplete).
 *                With a host array the call waits for its kernels, copies
 *                the two counters there and returns DPC_EOVERFLOW if the
 *                first is nonzero, DPC_ENOTSUP if the second is.
 * nloc = 0 is a no-op.  Errors and ownership as the calls above.            */
int dpc_nlist_build(void* stream, int nloc, int ntypes, const int* sel, double box, double rc,
                    const double* coord, const int* atype, void* workspace,
                    size_t workspace_bytes, int* nlist, int* status_host);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): dpc_nlist_build
 * with its cell list kept in a static device array of the library instead of
 * a caller's workspace.  The call allocates nothing and never waits.  Each
 * GPU it runs on holds one copy of that array (about 25 MB: the layout for
 * DPC_NLIST_NOALLOC_MAX_ATOMS atoms) until the process ends.
 *   nloc    at most DPC_NLIST_NOALLOC_MAX_ATOMS (else DPC_ENOTSUP)
 *   stream  must run on the current device (else DPC_EINVAL)
 *   status  device out int [2] or NULL: the two counters of dpc_nlist_build
 *           (truncated lists, lists over capacity), written by the kernels
 * All calls on one GPU share the array and every call starts by clearing
 * its counters and overwrites the rest: calls that overlap in time on one
 * GPU (other streams, other host threads) race, and the caller must
 * serialise them.  Other arguments, results and errors as dpc_nlist_build. */
#define DPC_NLIST_NOALLOC_MAX_ATOMS 524288
int dpc_nlist_build_noalloc(void* stream, int nloc, int ntypes, const int* sel, double box,
                            double rc, const double* coord, const int* atype, int* nlist,
                            int* status);

/* Forces and per-atom virials from dE/dR~ (F = -dE/dr; paper Sec. II: the
 * forces need the derivatives of E with respect to R~).  With
 * g_is = dE/dr_ij = sum_c dE/dR~_is[c] dR~_is[c]/dr_ij (dR~/dr from the
 * positions, as in dpc_env_mat_a):
 *   force[i]  = sum_s g_is - sum_s g_{j, rev[i][s]}   (j = nlist[i][s])
 *   virial[i] = -sum_s r_is (x) g_is   (row-major 3x3: [a][b] = -sum r_a g_b)
 * so that a neighbour list in which every pair within rc appears in both
 * atoms' lists (no sel truncation) gives F = -dE/dr for every atom, and the
 * summed virial is -dE/d(eps) of the homogeneous strain r_ij -> (1+eps) r_ij
 * (transposed).  Each atom gathers its terms in a fixed order: the result is
 * bitwise reproducible.
 *   dE_dem  device [nloc][nnei][4]: float32 for DPC_F32, float64 otherwise
 *   rev     from dpc_nlist_reverse for this nlist
 *   force   device out float64 [nloc][3]; virial device out float64 [nloc][9] or NULL
 * Other arguments as dpc_env_mat_a.  Arithmetic is float64.                 */
int dpc_force_a(void* stream, dpc_dtype dtype, int nloc, int ntypes, int nnei, double box,
                double rc, double rcs, const double* sigma, const double* sigma_all,
                const double* coord, const int* atype, const int* nlist, const int* rev,
                const void* dE_dem, double* force, double* virial);

/* Fitting net (paper Sec. II: a fully connected network maps the descriptor
 * D_i to the atomic energy E_i; Sec. III: widths (240, 240, 240)), read as
 *   h_1 = tanh(x W_1 + b_1),  h_l = h_{l-1} + tanh(h_{l-1} W_l + b_l) (l = 2, 3),
 *   E_i = h_3 . w_out + b_out,   x = D_i flattened row-major (n_in = m1 * m2),
 * with its backward dE_i/dD_i (the dE_dD input of dpc_descriptor_bwd).
 * Weights are device float64, row-major: W[0] [n_in][width], W[1], W[2]
 * [width][width], b[l] [width], w_out [width]; the three widths are equal.  */
typedef struct {
  int n_in, width;
  const double* W[3];
  const double* b[3];
  const double* w_out;
  double b_out;
} dpc_fitting_net;

/* Bytes of device workspace dpc_fitting_fwd_bwd needs: five float64 arrays
 * of nloc * width (rounded up to even) elements: the tanh outputs of layers
 * 1 and 2, h_2, the pre-activations and the backward accumulator.
 * 0 for bad sizes.                                                         */
size_t dpc_fitting_workspace_bytes(int nloc, int width);

/* E [nloc] and, if dE_dD is not NULL, dE/dD [nloc][n_in] (float64) for
 * D [nloc][n_in] (float64, device).  The layer products run as rocBLAS
 * double-precision GEMMs on the caller's handle `blas` (a rocblas_handle as
 * void*; its stream is left set to `stream`; its pointer mode is host for
 * the call and restored after it);
 * this library allocates nothing: `workspace` (device, 16-byte aligned,
 * >= dpc_fitting_workspace_bytes) is the caller's (rocBLAS may keep a
 * workspace of its own inside the handle).  Sums have a fixed order
 * for a given rocBLAS.  DPC_EHIP reports a HIP or rocBLAS failure.          */
int dpc_fitting_fwd_bwd(void* stream, void* blas, int nloc, const dpc_fitting_net* net,
                        const double* D, void* workspace, size_t workspace_bytes, double* E,
                        double* dE_dD);

#ifdef __cplusplus
}
#endif
#endif /* DPC_H */

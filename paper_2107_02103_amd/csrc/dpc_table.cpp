// Host side of libdpc: status strings, coefficient layout and the table
// builder (DP Compress, arXiv:2107.02103, Sec. II).
//
// The builder evaluates the embedding net and its first two derivatives at
// every node in float64 (forward-mode propagation through the tanh layers),
// then fits on each interval the quintic in the local offset t = x - x_l that
// matches value, slope and curvature at both nodes (the paper's six
// constraints).  The coefficients are obtained by eliminating the three known
// low-order terms first:
//     f = y_l,  e = y'_l,  d = y''_l / 2,
//     A = y_{l+1} - y_l - y'_l dt - y''_l dt^2 / 2
//     B = y'_{l+1} - y'_l - y''_l dt
//     C = y''_{l+1} - y''_l
// after which the 3x3 system for (a dt^5, b dt^4, c dt^3) has the solution
//     a dt^5 = 6A - 3B dt + C dt^2 / 2
//     b dt^4 = -15A + 7B dt - C dt^2
//     c dt^3 = 10A - 4B dt + C dt^2 / 2,
// which expands to the paper's closed forms for a, b and c.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#include "dpc.h"

extern "C" const char* dpc_strerror(int status) {
  switch (status) {
    case DPC_OK: return "ok";
    case DPC_EINVAL: return "invalid argument (null pointer, size, shape or dtype)";
    case DPC_ERANGE: return "invalid table range (stride <= 0, interval count < 1 or non-finite bound)";
    case DPC_EHIP: return "HIP runtime or kernel launch error";
    case DPC_ENOTSUP: return "unsupported size (m1 > 256, more than 8 atom types, more atoms within r_c than a list can hold, or more atoms than the no-allocation neighbour list holds)";
    case DPC_EOVERFLOW: return "neighbour list truncated: more atoms of some type within r_c than sel allows";
    default: return "unknown status";
  }
}

extern "C" int dpc_version(void) { return 100; }  // 0.1.0

namespace {

bool range_ok(const dpc_range& r) {
  return std::isfinite(r.lo) && std::isfinite(r.d1) && std::isfinite(r.d2) && r.d1 > 0.0 &&
         r.d2 > 0.0 && r.L1 >= 1 && r.L2 >= 1 && r.L1 < (int64_t(1) << 26) &&
         r.L2 < (int64_t(1) << 26);
}

size_t dtype_bytes(dpc_dtype dt) { return dt == DPC_F64 ? 8 : 4; }

bool dtype_ok(int dt) { return dt == DPC_F64 || dt == DPC_F32 || dt == DPC_F32_ACC64; }

// Value, first and second derivative of every output channel at input x.
struct NetEval {
  const dpc_net& net;
  std::vector<double> y, dy, d2y, ny, ndy, nd2y;
  explicit NetEval(const dpc_net& n) : net(n) {}

  void run(double x) {
    y.assign(1, x);
    dy.assign(1, 1.0);
    d2y.assign(1, 0.0);
    for (int k = 0; k < net.n_layers; ++k) {
      const int fi = net.widths[k], fo = net.widths[k + 1];
      const double* W = net.W[k];
      const double* b = net.b[k];
      ny.assign(fo, 0.0);
      ndy.assign(fo, 0.0);
      nd2y.assign(fo, 0.0);
      for (int o = 0; o < fo; ++o) {
        double z = b[o], z1 = 0.0, z2 = 0.0;
        for (int i = 0; i < fi; ++i) {
          const double w = W[(size_t)i * fo + o];
          z += y[i] * w;
          z1 += dy[i] * w;
          z2 += d2y[i] * w;
        }
        const double th = std::tanh(z);
        const double s = 1.0 - th * th;        // d tanh / dz
        double v = th, v1 = s * z1, v2 = s * z2 - 2.0 * th * s * z1 * z1;
        if (fo == 2 * fi) {                    // residual: input concatenated twice
          v += y[o % fi];
          v1 += dy[o % fi];
          v2 += d2y[o % fi];
        } else if (fo == fi) {                 // residual: identity
          v += y[o];
          v1 += dy[o];
          v2 += d2y[o];
        }
        ny[o] = v;
        ndy[o] = v1;
        nd2y[o] = v2;
      }
      y.swap(ny);
      dy.swap(ndy);
      d2y.swap(nd2y);
    }
  }
};

template <typename T>
void fit_segment(const double* y0, const double* y0p, const double* y0pp, const double* y1,
                 const double* y1p, const double* y1pp, double dt, int m1, int ld, T* out) {
  const double dt2 = dt * dt, dt3 = dt2 * dt, dt4 = dt3 * dt, dt5 = dt4 * dt;
  for (int m = 0; m < m1; ++m) {
    const double A = y1[m] - y0[m] - y0p[m] * dt - 0.5 * y0pp[m] * dt2;
    const double B = y1p[m] - y0p[m] - y0pp[m] * dt;
    const double C = y1pp[m] - y0pp[m];
    const double a = (6.0 * A - 3.0 * B * dt + 0.5 * C * dt2) / dt5;
    const double b = (-15.0 * A + 7.0 * B * dt - C * dt2) / dt4;
    const double c = (10.0 * A - 4.0 * B * dt + 0.5 * C * dt2) / dt3;
    // the coefficients of t^(2j) and t^(2j+1) of one channel are adjacent
    out[DPC_TABLE_AT(ld, 0, m)] = (T)y0[m];
    out[DPC_TABLE_AT(ld, 1, m)] = (T)y0p[m];
    out[DPC_TABLE_AT(ld, 2, m)] = (T)(0.5 * y0pp[m]);
    out[DPC_TABLE_AT(ld, 3, m)] = (T)c;
    out[DPC_TABLE_AT(ld, 4, m)] = (T)b;
    out[DPC_TABLE_AT(ld, 5, m)] = (T)a;
  }
  for (int q = 0; q < 6; ++q)
    for (int m = m1; m < ld; ++m) out[DPC_TABLE_AT(ld, q, m)] = (T)0;
}

template <typename T>
void build(const dpc_net& net, const dpc_range& r, T* out) {
  const int m1 = net.widths[net.n_layers];
  const int ld = DPC_TABLE_LD(m1);
  NetEval ev(net);
  std::vector<double> py, pdy, pd2y;
  const double x_up = r.lo + (double)r.L1 * r.d1;
  int64_t l = 0;
  for (int seg = 0; seg < 2; ++seg) {
    const double x0 = seg == 0 ? r.lo : x_up;
    const double dt = seg == 0 ? r.d1 : r.d2;
    const int64_t n = seg == 0 ? r.L1 : r.L2;
    ev.run(x0);
    py = ev.y;
    pdy = ev.dy;
    pd2y = ev.d2y;
    for (int64_t q = 1; q <= n; ++q, ++l) {
      ev.run(x0 + (double)q * dt);
      fit_segment<T>(py.data(), pdy.data(), pd2y.data(), ev.y.data(), ev.dy.data(),
                     ev.d2y.data(), dt, m1, ld, out + (size_t)l * 6 * ld);
      py.swap(ev.y);
      pdy.swap(ev.dy);
      pd2y.swap(ev.d2y);
    }
  }
}

}  // namespace

extern "C" int dpc_table_layout(int npair, int m1, dpc_range* ranges, dpc_dtype dtype,
                                size_t* total_bytes) {
  if (npair < 1 || m1 < 1 || !ranges || !total_bytes || !dtype_ok(dtype)) return DPC_EINVAL;
  if (m1 > DPC_MAX_M1 || npair > DPC_MAX_TYPES * DPC_MAX_TYPES) return DPC_ENOTSUP;
  int64_t off = 0;
  for (int p = 0; p < npair; ++p)
    if (!range_ok(ranges[p])) return DPC_ERANGE;
  for (int p = 0; p < npair; ++p) {
    ranges[p].offset = off;
    off += (ranges[p].L1 + ranges[p].L2) * 6 * (int64_t)DPC_TABLE_LD(m1);
  }
  if (off >= (int64_t(1) << 31)) return DPC_ENOTSUP;  // kernels index with 32-bit offsets
  *total_bytes = (size_t)off * dtype_bytes(dtype);
  return DPC_OK;
}

extern "C" int dpc_build_table(const dpc_net* net, const dpc_range* range, dpc_dtype dtype,
                               void* host_out) {
  if (!net || !range || !host_out || !dtype_ok(dtype) || net->n_layers < 1 || !net->widths ||
      !net->W || !net->b)
    return DPC_EINVAL;
  if (net->widths[0] != 1) return DPC_EINVAL;
  for (int k = 0; k < net->n_layers; ++k)
    if (net->widths[k + 1] < 1 || !net->W[k] || !net->b[k]) return DPC_EINVAL;
  if (net->widths[net->n_layers] > DPC_MAX_M1) return DPC_ENOTSUP;
  if (!range_ok(*range)) return DPC_ERANGE;
  if (dtype == DPC_F64)
    build<double>(*net, *range, static_cast<double*>(host_out));
  else
    build<float>(*net, *range, static_cast<float*>(host_out));
  return DPC_OK;
}

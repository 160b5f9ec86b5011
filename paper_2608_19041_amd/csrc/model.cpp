// Model creation: blob parsing, radial tabulation, Gaunt couplings and the
// device-resident parameter block (Methods "Compressed inference").
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <memory>
#include <vector>

#include "../../include/dpa4c.h"
#include "launch.h"
#include "model.h"

namespace dpa4c {

int DevBuf::ensure(size_t want) {
  if (want <= bytes && p) return 0;
  if (p) {
    hipFree(p);
    p = nullptr;
    bytes = 0;
  }
  size_t b = want < 256 ? 256 : want;
  // Large requests keep a reserve of device memory free for the runtime
  // (kernel scratch, the caller's own allocations): running the device to the
  // last byte can make a later, unrelated call fail.  Such a request reports
  // out-of-memory like a failed hipMalloc.
  constexpr size_t kReserve = size_t(512) << 20;
  if (b > (size_t(64) << 20)) {
    size_t free_b = 0, total_b = 0;
    if (hipMemGetInfo(&free_b, &total_b) == hipSuccess && b + kReserve > free_b) {
      set_error("allocation of " + std::to_string(b) + " bytes would leave less than 512 MiB of " +
                std::to_string(free_b) + " bytes of device memory free");
      return DPA4C_ERR_OOM;
    }
  }
  hipError_t e = hipMalloc(&p, b);
  if (e != hipSuccess) {
    p = nullptr;
    set_error(std::string("hipMalloc of ") + std::to_string(b) + " bytes: " + hipGetErrorString(e));
    return e == hipErrorOutOfMemory ? DPA4C_ERR_OOM : DPA4C_ERR_HIP;
  }
  bytes = b;
  return 0;
}

void DevBuf::release() {
  if (p) hipFree(p);
  p = nullptr;
  bytes = 0;
}

const char* stage_name(int s) {
  static const char* names[kNumStages] = {"neighbor", "skin_rev", "forward", "atoms",
                                          "backward", "forces",   "energy",  "integrate"};
  return (s >= 0 && s < kNumStages) ? names[s] : "?";
}

namespace {

// ---------------------------------------------------------------------------
// real Cartesian harmonics on the unit sphere (s = |u|^2 = 1), degrees 1..4,
// Eq. (harmonics) and the degree-three and degree-four blocks of the
// Supplementary Note
// ---------------------------------------------------------------------------
void harmonics_host(int l, double x, double y, double z, double* out) {
  const double r3 = std::sqrt(3.0);
  if (l == 1) {
    out[0] = x; out[1] = y; out[2] = z;
  } else if (l == 2) {
    out[0] = r3 * x * y;
    out[1] = r3 * y * z;
    out[2] = 0.5 * (3 * z * z - 1.0);
    out[3] = r3 * x * z;
    out[4] = 0.5 * r3 * (x * x - y * y);
  } else if (l == 3) {
    out[0] = std::sqrt(5.0 / 8.0) * y * (3 * x * x - y * y);
    out[1] = std::sqrt(15.0) * x * y * z;
    out[2] = std::sqrt(3.0 / 8.0) * y * (5 * z * z - 1.0);
    out[3] = 0.5 * z * (5 * z * z - 3.0);
    out[4] = std::sqrt(3.0 / 8.0) * x * (5 * z * z - 1.0);
    out[5] = 0.5 * std::sqrt(15.0) * z * (x * x - y * y);
    out[6] = std::sqrt(5.0 / 8.0) * x * (x * x - 3 * y * y);
  } else {
    const double x2 = x * x, y2 = y * y, z2 = z * z;
    out[0] = 0.5 * std::sqrt(35.0) * x * y * (x2 - y2);
    out[1] = 0.25 * std::sqrt(70.0) * y * z * (3 * x2 - y2);
    out[2] = 0.5 * std::sqrt(5.0) * x * y * (7 * z2 - 1.0);
    out[3] = 0.25 * std::sqrt(10.0) * y * z * (7 * z2 - 3.0);
    out[4] = 0.125 * (35 * z2 * z2 - 30 * z2 + 3.0);
    out[5] = 0.25 * std::sqrt(10.0) * x * z * (7 * z2 - 3.0);
    out[6] = 0.25 * std::sqrt(5.0) * (x2 - y2) * (7 * z2 - 1.0);
    out[7] = 0.25 * std::sqrt(70.0) * x * z * (x2 - 3 * y2);
    out[8] = 0.125 * std::sqrt(35.0) * (x2 * x2 - 6 * x2 * y2 + y2 * y2);
  }
}

// Gauss-Legendre nodes and weights on [-1, 1] by Newton iteration.
void gauss_legendre(int n, std::vector<double>& x, std::vector<double>& w) {
  x.resize(n);
  w.resize(n);
  for (int i = 0; i < n; ++i) {
    double t = std::cos(M_PI * (i + 0.75) / (n + 0.5));
    for (int it = 0; it < 100; ++it) {
      double p0 = 1.0, p1 = t;
      for (int k = 2; k <= n; ++k) {
        double p2 = ((2 * k - 1) * t * p1 - (k - 1) * p0) / k;
        p0 = p1;
        p1 = p2;
      }
      double dp = n * (t * p1 - p0) / (t * t - 1.0);
      double dt = p1 / dp;
      t -= dt;
      if (std::fabs(dt) < 1e-16) break;
    }
    double p0 = 1.0, p1 = t;
    for (int k = 2; k <= n; ++k) {
      double p2 = ((2 * k - 1) * t * p1 - (k - 1) * p0) / k;
      p0 = p1;
      p1 = p2;
    }
    double dp = n * (t * p1 - p0) / (t * t - 1.0);
    x[i] = t;
    w[i] = 2.0 / ((1.0 - t * t) * dp * dp);
  }
}

// Eq. (gaunt): I = integral of B_l1 B_l2 B_l3 over the unit sphere, exact
// for the degree-<=12 polynomial integrand with 10 x 26 product nodes;
// returned normalised as C = -I / ||I||_F (the sign convention that gives
// the closed forms of Eq. (closed-forms)).
std::vector<double> coupling(int l1, int l2, int l3) {
  std::vector<double> zx, zw;
  gauss_legendre(10, zx, zw);
  const int nphi = 26;
  int n1 = 2 * l1 + 1, n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
  std::vector<double> I(n1 * n2 * n3, 0.0);
  double b1[9], b2[9], b3[9];
  for (size_t a = 0; a < zx.size(); ++a) {
    double z = zx[a], st = std::sqrt(1.0 - z * z);
    for (int p = 0; p < nphi; ++p) {
      double ph = 2.0 * M_PI * p / nphi;
      double x = st * std::cos(ph), y = st * std::sin(ph);
      double wt = zw[a] * 2.0 * M_PI / nphi;
      harmonics_host(l1, x, y, z, b1);
      harmonics_host(l2, x, y, z, b2);
      harmonics_host(l3, x, y, z, b3);
      for (int i = 0; i < n1; ++i)
        for (int j = 0; j < n2; ++j)
          for (int k = 0; k < n3; ++k) I[(i * n2 + j) * n3 + k] += wt * b1[i] * b2[j] * b3[k];
    }
  }
  double nrm = 0;
  for (double v : I) nrm += v * v;
  nrm = std::sqrt(nrm);
  for (double& v : I) v = -v / nrm;
  return I;
}

// ---------------------------------------------------------------------------
// Radial map [g, q](rho) with its first two derivatives, float64.
// Eqs. (bessel-basis), (swiglu), (radial-map), (radial-modes).
// ---------------------------------------------------------------------------
struct RadialNet {
  int n_rbf, H, C0, R;
  const float *omega, *W_in, *W_out, *W_mode;

  void jet(double rho, double* y0, double* y1, double* y2) const {
    std::vector<double> f(n_rbf), f1(n_rbf), f2(n_rbf);
    for (int n = 0; n < n_rbf; ++n) {
      double w = omega[n], x = w * rho;
      if (std::fabs(x) < 1.0) {
        // Taylor series of sin(x)/x and its derivatives (|x| < 1)
        double s0 = 0, s1 = 0, s2 = 0, fact = 1.0;   // fact = (2k+1)!
        double xp = 1.0;                             // x^(2k)
        double xprev = 0.0;                          // x^(2k-2)
        for (int k = 0; k <= 12; ++k) {
          if (k > 0) fact *= (2.0 * k) * (2.0 * k + 1.0);
          double sg = (k % 2) ? -1.0 : 1.0;
          s0 += sg * xp / fact;
          if (k >= 1) {
            s1 += sg * 2.0 * k * (xprev * x) / fact;                 // x^(2k-1)
            s2 += sg * 2.0 * k * (2.0 * k - 1.0) * xprev / fact;     // x^(2k-2)
          }
          xprev = xp;
          xp *= x * x;
        }
        f[n] = w * s0;
        f1[n] = w * w * s1;
        f2[n] = w * w * w * s2;
      } else {
        double s = std::sin(x), c = std::cos(x);
        f[n] = s / rho;
        f1[n] = w * c / rho - s / (rho * rho);
        f2[n] = -w * w * s / rho - 2.0 * w * c / (rho * rho) + 2.0 * s / (rho * rho * rho);
      }
    }
    std::vector<double> h(H), h1(H), h2(H);
    for (int k = 0; k < H; ++k) {
      double a = 0, a1 = 0, a2 = 0, b = 0, b1 = 0, b2 = 0;
      for (int n = 0; n < n_rbf; ++n) {
        double wa = W_in[n * 2 * H + k], wb = W_in[n * 2 * H + H + k];
        a += f[n] * wa; a1 += f1[n] * wa; a2 += f2[n] * wa;
        b += f[n] * wb; b1 += f1[n] * wb; b2 += f2[n] * wb;
      }
      double sg = 1.0 / (1.0 + std::exp(-a));
      double s0 = a * sg;
      double sd1 = sg * (1.0 + a * (1.0 - sg));
      double sd2 = sg * (1.0 - sg) * (2.0 + a * (1.0 - 2.0 * sg));
      h[k] = s0 * b;
      h1[k] = sd1 * a1 * b + s0 * b1;
      h2[k] = sd2 * a1 * a1 * b + sd1 * a2 * b + 2.0 * sd1 * a1 * b1 + s0 * b2;
    }
    for (int c = 0; c < C0 + R; ++c) {
      double v0 = 0, v1 = 0, v2 = 0;
      for (int k = 0; k < H; ++k) {
        double w = c < C0 ? W_out[k * C0 + c] : W_mode[k * R + (c - C0)];
        v0 += h[k] * w; v1 += h1[k] * w; v2 += h2[k] * w;
      }
      y0[c] = v0; y1[c] = v1; y2[c] = v2;
    }
  }
};

// Normalised quintic Hermite coefficients (Supplementary Note "Quintic
// Hermite interpolation"): ctilde_n = c_n Delta^n on [rho_s, rho_s + Delta].
void quintic(double d, double y0, double p0, double q0, double y1, double p1, double q1,
             double* c) {
  double dl = y1 - y0;
  c[0] = y0;
  c[1] = p0 * d;
  c[2] = 0.5 * q0 * d * d;
  c[3] = 0.5 * (20.0 * dl - (8.0 * p1 + 12.0 * p0) * d - (3.0 * q0 - q1) * d * d);
  c[4] = 0.5 * (-30.0 * dl + (14.0 * p1 + 16.0 * p0) * d + (3.0 * q0 - 2.0 * q1) * d * d);
  c[5] = 0.5 * (12.0 * dl - 6.0 * (p1 + p0) * d + (q1 - q0) * d * d);
}

struct Reader {
  const uint8_t* p;
  size_t left;
  const float* take(size_t n) {
    if (n * 4 > left) return nullptr;
    const float* r = reinterpret_cast<const float*>(p);
    p += n * 4;
    left -= n * 4;
    return r;
  }
};

}  // namespace

// The header checks, on the host only: magic, version, a compiled profile
// and sane values.  Fills the header fields of ``m`` and the widths.
int read_header(const void* blob, size_t nbytes, dpa4c_model* m, int widths[2]) {
  if (!blob || nbytes < 64) {
    set_error("dpa4c_model_create: null blob/out or blob shorter than its header");
    return DPA4C_ERR_INVALID_ARG;
  }
  const uint8_t* b = static_cast<const uint8_t*>(blob);
  if (std::memcmp(b, "DPA4CW01", 8) != 0) {
    set_error("dpa4c_model_create: bad magic");
    return DPA4C_ERR_INVALID_ARG;
  }
  int32_t hdr[8];
  std::memcpy(hdr, b + 8, 32);
  double rc_delta[2];
  std::memcpy(rc_delta, b + 40, 16);
  if (hdr[0] != 1) {
    set_error("dpa4c_model_create: unknown blob version");
    return DPA4C_ERR_INVALID_ARG;
  }
  m->C0 = hdr[1]; m->L = hdr[2]; m->R = hdr[3]; m->n_rbf = hdr[4];
  m->F = hdr[5]; m->n_layers = hdr[6]; m->n_types = hdr[7];
  m->r_c = rc_delta[0];
  m->delta = rc_delta[1];
  if (with_profile(m->C0, m->L, m->R, m->F, [&](auto p, auto) {
        widths[0] = decltype(p)::S;
        widths[1] = decltype(p)::DOUT;
        return 0;
      }) == kNoProfile) {
    set_error("dpa4c_model_create: (C0, L, R, MLP width) is not one of the compiled variants "
              "(8,2,0,96) (32,2,0,192) (64,2,0,256) (64,3,4,256) (128,3,4,384) (128,4,4,384)");
    return DPA4C_ERR_UNSUPPORTED;
  }
  if (m->n_rbf <= 0 || m->F <= 0 || m->F % 16 || m->n_layers < 1 || m->n_layers > 7 ||
      m->n_types <= 0 || !(m->r_c > 0) || !(m->delta > 0) || m->r_c / m->delta > 1e6) {
    set_error("dpa4c_model_create: bad header values");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (m->n_types + 1 > kMaxTypeRows) {   // the per-call species bitmask has 128 bits
    set_error("dpa4c_model_create: more than 127 species (the type table holds at most 128 rows)");
    return DPA4C_ERR_UNSUPPORTED;
  }
  return 0;
}

int check_blob_header(const void* blob, size_t nbytes) {
  dpa4c_model m;
  int widths[2] = {0, 0};
  return read_header(blob, nbytes, &m, widths);
}

int create_model(const void* blob, size_t nbytes, int device, dpa4c_model** out) {
  if (!out) {
    set_error("dpa4c_model_create: null blob/out or blob shorter than its header");
    return DPA4C_ERR_INVALID_ARG;
  }
  std::unique_ptr<dpa4c_model> m(new dpa4c_model());
  m->device = device;
  int widths[2] = {0, 0};   // S, D_out of the compiled profile
  if (int rc = read_header(blob, nbytes, m.get(), widths)) return rc;
  const uint8_t* b = static_cast<const uint8_t*>(blob);
  const int C0 = m->C0, L = m->L, R = m->R, T1 = m->n_types + 1;
  auto ceil_log2 = [](int x) { int k = 0; while ((1 << k) < x) ++k; return k; };
  int C1 = std::max(4, 1 << ((ceil_log2(C0) + 1) / 2));
  int C2 = std::max(4, C1 / 2);
  m->C[0] = C0; m->C[1] = C1; m->C[2] = C2; m->C[3] = 1; m->C[4] = 1;
  m->K[1] = C2; m->K[2] = 2; m->K[3] = 1; m->K[4] = 1;
  m->S = widths[0];
  m->D_out = widths[1];
  m->H = 8 * ((C0 + 2) / 3);
  m->Hp = 8 * ((2 * C0 + 2) / 3);
  const int H = m->H, Hp = m->Hp, F = m->F, D = m->D_out, K1 = C2, K2 = 2;
  m->n_rows = static_cast<int>(std::ceil(m->r_c / m->delta - 1e-9));

  Reader rd{b + 64, nbytes - 64};
  const float* type_embed = rd.take(size_t(T1) * C0);
  const float* omega = rd.take(m->n_rbf);
  const float* W_in = rd.take(size_t(m->n_rbf) * 2 * H);
  const float* W_out = rd.take(size_t(H) * C0);
  const float* W_mode = rd.take(size_t(H) * R);
  const float* Wp_in = rd.take(size_t(2 * C0) * 2 * Hp);
  const float* Wp_out = rd.take(size_t(Hp) * C0 * (2 + R));
  const float* Wa1 = rd.take(size_t(C1) * C1);
  const float* Wa2 = rd.take(size_t(C2) * C2);
  const float* A1 = (K1 != C1) ? rd.take(size_t(C1) * K1) : nullptr;
  const float* A2 = rd.take(size_t(C2) * K2);
  const float* theta[8] = {};
  const float* bias[8] = {};
  int fan = D;
  for (int t = 0; t < m->n_layers; ++t) {
    theta[t] = rd.take(size_t(fan) * F);
    bias[t] = rd.take(F);
    fan = F;
  }
  const float* w_head = rd.take(F);
  const float* b_head = rd.take(1);
  const float* E_ref = rd.take(T1);
  const float* mu = rd.take(D);
  const float* sigma = rd.take(D);
  if (!sigma || rd.left != 0 || (K1 != C1 && !A1)) {
    set_error("dpa4c_model_create: blob size does not match its header");
    return DPA4C_ERR_INVALID_ARG;
  }
  for (int k = 0; k < D; ++k)
    if (!(sigma[k] != 0.0f) || !std::isfinite(sigma[k])) {
      set_error("dpa4c_model_create: calibration scale must be finite and nonzero");
      return DPA4C_ERR_INVALID_ARG;
    }

  // ---- radial table in the kernels' lane layout -------------------------
  const int LPE = C1, CPL = C0 / LPE, P = C0 + R, rows = m->n_rows;
  std::vector<float> gtab(size_t(rows) * C0 * 6), qtab(size_t(rows) * std::max(R, 1) * 6, 0.f);
  {
    RadialNet net{m->n_rbf, H, C0, R, omega, W_in, W_out, W_mode};
    std::vector<double> a0(P), a1(P), a2(P), b0(P), b1(P), b2(P);
    net.jet(0.0, a0.data(), a1.data(), a2.data());
    for (int s = 0; s < rows; ++s) {
      net.jet((s + 1) * m->delta, b0.data(), b1.data(), b2.data());
      for (int c = 0; c < P; ++c) {
        double co[6];
        quintic(m->delta, a0[c], a1[c], a2[c], b0[c], b1[c], b2[c], co);
        float* dst;
        if (c < C0) {
          int k = c % LPE, j = c / LPE;
          dst = &gtab[((size_t(s) * CPL + j) * LPE + k) * 6];
        } else {
          dst = &qtab[(size_t(s) * R + (c - C0)) * 6];
        }
        for (int q = 0; q < 6; ++q) dst[q] = static_cast<float>(co[q]);
      }
      std::swap(a0, b0); std::swap(a1, b1); std::swap(a2, b2);
    }
  }
  // float16 scales of the folded tables' c2, c3 (and of c4, c5, for the
  // bound): a power of two that maps the bound 2 max|g_n| + R max|q_n|
  // (gamma = 1 + tanh < 2, |U| = |tanh| < 1) to at most 2^14, half of the
  // float16 range.  The rounding of c2, c3 (at most 2^-11 of each bound)
  // enters the value with weight 1 and d/dtau with weights 2, 3; c4 and c5
  // are dropped, so their whole bounds enter with weights 1 and 4, 5.  The
  // tables are folded only while the value error stays below the float32
  // rounding of the value term c0 and the slope error below 2^-14 of the
  // slope term c1, else the separable float32 tables are used.
  double bnd[6] = {};
  for (int q = 0; q < 6; ++q) {
    double gmax = 0.0, qmax = 0.0;
    for (size_t e = q; e < gtab.size(); e += 6) gmax = std::max(gmax, double(std::fabs(gtab[e])));
    for (size_t e = q; e < qtab.size(); e += 6) qmax = std::max(qmax, double(std::fabs(qtab[e])));
    bnd[q] = 2.0 * gmax + double(R) * qmax;
  }
  for (int q = 2; q < 6; ++q) {
    int ex = 0;
    if (bnd[q] > 0.0) ex = static_cast<int>(std::floor(std::log2(16384.0 / bnd[q])));
    ex = std::max(-100, std::min(100, ex));
    m->c_scale[q - 2] = static_cast<float>(std::ldexp(1.0, ex));
  }
  const double f16 = std::ldexp(1.0, -11);
  const double val_lim = bnd[0] * std::ldexp(1.0, -24), slope_lim = bnd[1] * std::ldexp(1.0, -14);
  m->fold_allowed = (bnd[2] + bnd[3]) * f16 + bnd[4] + bnd[5] <= val_lim &&
                    (2.0 * bnd[2] + 3.0 * bnd[3]) * f16 + 4.0 * bnd[4] + 5.0 * bnd[5] <= slope_lim;

  // ---- coupling tensors, each symmetrised over the indices of equal degree
  // (the exact integrals are; the quadrature sums are only up to rounding)
  std::vector<float> cpl;
  m->gaunt[0] = coupling(1, 1, 2);
  m->gaunt[2] = coupling(2, 2, 2);
  auto push = [&](int l1, int l2, int l3) {
    const std::vector<double> g = coupling(l1, l2, l3);
    const int n1 = 2 * l1 + 1, n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
    auto at = [&](int a, int b, int c) { return g[(a * n2 + b) * n3 + c]; };
    for (int a = 0; a < n1; ++a)
      for (int b = 0; b < n2; ++b)
        for (int c = 0; c < n3; ++c) {
          double v;
          if (l1 == l2 && l2 == l3)
            v = (at(a, b, c) + at(a, c, b) + at(b, a, c) + at(b, c, a) + at(c, a, b) + at(c, b, a)) / 6.0;
          else if (l2 == l3)
            v = 0.5 * (at(a, b, c) + at(a, c, b));
          else if (l1 == l2)
            v = 0.5 * (at(a, b, c) + at(b, a, c));
          else
            v = at(a, b, c);
          cpl.push_back(static_cast<float>(v));
        }
  };
  if (L >= 3) {
    cpl.reserve(couplings_for(L));
    push(1, 2, 3);
    push(2, 3, 3);
  }
  if (L >= 4) {
    push(1, 3, 4);
    push(2, 2, 4);
    push(2, 4, 4);
    push(3, 3, 4);
    push(4, 4, 4);
  }
  if (cpl.size() != size_t(couplings_for(L))) {
    set_error("dpa4c_model_create: coupling layout");
    return DPA4C_ERR_INVALID_ARG;
  }

  // ---- one device block for every parameter array ---------------------
  std::vector<float> inv_sigma(D);
  for (int k = 0; k < D; ++k) inv_sigma[k] = 1.0f / sigma[k];
  struct Piece { void** dst; const void* src; size_t bytes; };
  std::vector<Piece> pieces;
  std::vector<std::vector<float>> transposed(m->n_layers);
  auto add = [&](void** dst, const void* src, size_t bytes) { pieces.push_back({dst, src, bytes}); };
  add((void**)&m->gtab, gtab.data(), gtab.size() * 4);
  add((void**)&m->qtab, qtab.data(), qtab.size() * 4);
  add((void**)&m->type_embed, type_embed, size_t(T1) * C0 * 4);
  add((void**)&m->W1, Wa1, size_t(C1) * C1 * 4);
  add((void**)&m->W2, Wa2, size_t(C2) * C2 * 4);
  if (A1) add((void**)&m->A1, A1, size_t(C1) * K1 * 4);
  add((void**)&m->A2, A2, size_t(C2) * K2 * 4);
  add((void**)&m->mu, mu, size_t(D) * 4);
  add((void**)&m->inv_sigma, inv_sigma.data(), size_t(D) * 4);
  add((void**)&m->E_ref, E_ref, size_t(T1) * 4);
  // Theta_1 is padded with zero rows to a multiple of 16 input features (the
  // descriptor row stride); every Theta_t is also stored transposed for the
  // input-gradient products of the backward pass
  const int Dp = (D + 15) / 16 * 16;
  std::vector<std::vector<float>> padded(m->n_layers);
  fan = D;
  for (int t = 0; t < m->n_layers; ++t) {
    const int fin = t == 0 ? Dp : F;
    auto& fw = padded[t];
    fw.assign(size_t(fin) * F, 0.0f);
    for (int r = 0; r < fan; ++r)
      for (int c = 0; c < F; ++c) fw[size_t(r) * F + c] = theta[t][size_t(r) * F + c];
    add((void**)&m->theta[t], fw.data(), fw.size() * 4);
    auto& tr = transposed[t];
    tr.assign(size_t(fin) * F, 0.0f);
    for (int r = 0; r < fan; ++r)
      for (int c = 0; c < F; ++c) tr[size_t(c) * fin + r] = theta[t][size_t(r) * F + c];
    add((void**)&m->thetaT[t], tr.data(), tr.size() * 4);
    add((void**)&m->bias[t], bias[t], size_t(F) * 4);
    fan = F;
  }
  // fragment order for the fused MLP kernel: for output tile T and k-block kb
  // lane l holds W[kb*16 + 4*(l/16) + s][T*16 + l%16], s = 0..3
  auto fragment = [](const std::vector<float>& src, int K, int N) {
    std::vector<float> out(size_t(K) * N);
    const int kbs = K / 16;
    for (int T = 0; T < N / 16; ++T)
      for (int kb = 0; kb < kbs; ++kb)
        for (int l = 0; l < 64; ++l)
          for (int s = 0; s < 4; ++s)
            out[((size_t(T) * kbs + kb) * 64 + l) * 4 + s] =
                src[size_t(kb * 16 + (l / 16) * 4 + s) * N + T * 16 + (l % 16)];
    return out;
  };
  std::vector<std::vector<float>> frags(2 * m->n_layers);
  for (int t = 0; t < m->n_layers; ++t) {
    const int fin = t == 0 ? Dp : F;
    frags[2 * t] = fragment(padded[t], fin, F);
    frags[2 * t + 1] = fragment(transposed[t], F, fin);
    add((void**)&m->wfrag[t], frags[2 * t].data(), frags[2 * t].size() * 4);
    add((void**)&m->wfragT[t], frags[2 * t + 1].data(), frags[2 * t + 1].size() * 4);
  }
  add((void**)&m->w_head, w_head, size_t(F) * 4);
  m->b_head = b_head[0];
  if (!cpl.empty()) add((void**)&m->cpl, cpl.data(), cpl.size() * 4);
  // raw pair-network weights, used once by the pair-cache kernel
  const float* raw_wp_in = nullptr;
  const float* raw_wp_out = nullptr;
  add((void**)&raw_wp_in, Wp_in, size_t(2 * C0) * 2 * Hp * 4);
  add((void**)&raw_wp_out, Wp_out, size_t(Hp) * C0 * (2 + R) * 4);
  size_t pair_bytes = size_t(T1) * T1 * C0 * (2 + R) * 4;
  size_t total = pair_bytes + 256;
  for (auto& pc : pieces) total += (pc.bytes + 255) / 256 * 256;

  DPA4C_HIP_TRY(hipSetDevice(device));
  DPA4C_TRY(m->params.ensure(total));
  std::vector<uint8_t> host(total - pair_bytes, 0);
  size_t off = 0;
  char* base = m->params.as<char>();
  m->pair = reinterpret_cast<float*>(base);
  off = (pair_bytes + 255) / 256 * 256;
  size_t hoff = 0;
  size_t first = off;
  for (auto& pc : pieces) {
    std::memcpy(host.data() + hoff, pc.src, pc.bytes);
    *pc.dst = base + off;
    size_t step = (pc.bytes + 255) / 256 * 256;
    off += step;
    hoff += step;
  }
  DPA4C_HIP_TRY(hipMemcpy(base + first, host.data(), hoff, hipMemcpyHostToDevice));
  int rc = launch_pair_cache(m.get(), raw_wp_in, raw_wp_out);
  if (rc) return rc;
  DPA4C_HIP_TRY(hipDeviceSynchronize());
  *out = m.release();
  return 0;
}

}  // namespace dpa4c

dpa4c::ModelDev dpa4c_model::dev() const {
  dpa4c::ModelDev d{};
  d.gtab = gtab;
  d.qtab = qtab;
  d.n_rows = n_rows;
  d.inv_delta = static_cast<float>(1.0 / delta);
  d.r_c = static_cast<float>(r_c);
  d.inv_rc = static_cast<float>(1.0 / r_c);
  d.n_types1 = n_types + 1;
  d.pair = pair;
  d.type_embed = type_embed;
  d.W1 = W1;
  d.W2 = W2;
  d.A1 = A1;
  d.A2 = A2;
  d.mu = mu;
  d.inv_sigma = inv_sigma;
  d.cpl = cpl;
  d.E_ref = E_ref;
  d.ftab = ws.ftab.as<float>();
  d.fold_n = fold_n > 0 ? fold_n : 0;
  for (int q = 0; q < 4; ++q) d.c_inv[q] = 1.0f / c_scale[q];
  return d;
}

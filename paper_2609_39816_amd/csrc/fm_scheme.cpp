// Host-side scheme handling for libfm: loading and validation, Kronecker
// power, gauge action, fp32 coefficient tables and the kernels' coefficient
// lists.  All arithmetic is float64, in the order stated at each function,
// so the tables are reproducible bit for bit (the file is built with
// -ffp-contract=off).
#include <cmath>
#include <cstring>

#include "fm_internal.h"

namespace fm {

// Largest violation of the Brent equations
//   sum_r u_{r,il} v_{r,l'j} w_{r,i'j'} = [i=i'][l=l'][j=j'],
// the condition for eq. (1) (Sec. 2.1) to compute AB for all A, B.
double brent_residual(const fm_scheme& s) {
  const int MK = s.m * s.k, KN = s.k * s.n, MN = s.m * s.n;
  double worst = 0.0;
  std::vector<double> acc((size_t)MK * KN * MN, 0.0);
  for (int r = 0; r < s.R; ++r) {
    const double* u = &s.U[(size_t)r * MK];
    const double* v = &s.V[(size_t)r * KN];
    const double* w = &s.W[(size_t)r * MN];
    for (int a = 0; a < MK; ++a) {
      if (u[a] == 0.0) continue;
      for (int b = 0; b < KN; ++b) {
        if (v[b] == 0.0) continue;
        const double uv = u[a] * v[b];
        double* row = &acc[((size_t)a * KN + b) * MN];
        for (int c = 0; c < MN; ++c) row[c] += uv * w[c];
      }
    }
  }
  for (int i = 0; i < s.m; ++i)
    for (int l = 0; l < s.k; ++l)
      for (int l2 = 0; l2 < s.k; ++l2)
        for (int j = 0; j < s.n; ++j)
          for (int i2 = 0; i2 < s.m; ++i2)
            for (int j2 = 0; j2 < s.n; ++j2) {
              const double want = (i == i2 && l == l2 && j == j2) ? 1.0 : 0.0;
              const double got =
                  acc[((size_t)(i * s.k + l) * KN + (l2 * s.n + j)) * MN + (i2 * s.n + j2)];
              worst = std::fmax(worst, std::fabs(got - want));
            }
  return worst;
}

// Scheme b applied inside every block of scheme a (a is the outer level):
// product r = ra*Rb + rb, block row i = ia*mb + ib (and likewise l, j),
// coefficient = (outer coefficient) * (inner coefficient).
fm_scheme kron(const fm_scheme& a, const fm_scheme& b) {
  fm_scheme o;
  o.m = a.m * b.m;
  o.k = a.k * b.k;
  o.n = a.n * b.n;
  o.R = a.R * b.R;
  o.U.assign((size_t)o.R * o.m * o.k, 0.0);
  o.V.assign((size_t)o.R * o.k * o.n, 0.0);
  o.W.assign((size_t)o.R * o.m * o.n, 0.0);
  for (int ra = 0; ra < a.R; ++ra)
    for (int rb = 0; rb < b.R; ++rb) {
      const int r = ra * b.R + rb;
      for (int ia = 0; ia < a.m; ++ia)
        for (int ib = 0; ib < b.m; ++ib)
          for (int la = 0; la < a.k; ++la)
            for (int lb = 0; lb < b.k; ++lb)
              o.U[(size_t)r * o.m * o.k + (ia * b.m + ib) * o.k + (la * b.k + lb)] =
                  a.U[(size_t)ra * a.m * a.k + ia * a.k + la] *
                  b.U[(size_t)rb * b.m * b.k + ib * b.k + lb];
      for (int la = 0; la < a.k; ++la)
        for (int lb = 0; lb < b.k; ++lb)
          for (int ja = 0; ja < a.n; ++ja)
            for (int jb = 0; jb < b.n; ++jb)
              o.V[(size_t)r * o.k * o.n + (la * b.k + lb) * o.n + (ja * b.n + jb)] =
                  a.V[(size_t)ra * a.k * a.n + la * a.n + ja] *
                  b.V[(size_t)rb * b.k * b.n + lb * b.n + jb];
      for (int ia = 0; ia < a.m; ++ia)
        for (int ib = 0; ib < b.m; ++ib)
          for (int ja = 0; ja < a.n; ++ja)
            for (int jb = 0; jb < b.n; ++jb)
              o.W[(size_t)r * o.m * o.n + (ia * b.m + ib) * o.n + (ja * b.n + jb)] =
                  a.W[(size_t)ra * a.m * a.n + ia * a.n + ja] *
                  b.W[(size_t)rb * b.m * b.n + ib * b.n + jb];
    }
  return o;
}

// The scheme applied `levels` times: ((s (x) s) (x) s) ..., outer level first.
fm_scheme power(const fm_scheme& s, int levels) {
  fm_scheme o = s;
  for (int l = 1; l < levels; ++l) o = kron(o, s);
  return o;
}

// Inverse of an n x n row-major matrix.  n <= 3: adjugate over the
// determinant (cofactor expansion along the first row); larger n:
// Gauss-Jordan elimination with partial pivoting (first row of largest
// magnitude wins a tie).
bool invert(const std::vector<double>& P, int n, std::vector<double>& out) {
  out.assign((size_t)n * n, 0.0);
  if (n == 1) {
    if (P[0] == 0.0) return false;
    out[0] = 1.0 / P[0];
    return true;
  }
  if (n == 2) {
    const double a = P[0], b = P[1], c = P[2], d = P[3];
    const double det = a * d - b * c;
    if (det == 0.0) return false;
    out[0] = d / det;
    out[1] = -b / det;
    out[2] = -c / det;
    out[3] = a / det;
    return true;
  }
  if (n == 3) {
    const double a = P[0], b = P[1], c = P[2];
    const double d = P[3], e = P[4], f = P[5];
    const double g = P[6], h = P[7], i = P[8];
    const double c00 = e * i - f * h;
    const double c01 = -(d * i - f * g);
    const double c02 = d * h - e * g;
    const double c10 = -(b * i - c * h);
    const double c11 = a * i - c * g;
    const double c12 = -(a * h - b * g);
    const double c20 = b * f - c * e;
    const double c21 = -(a * f - c * d);
    const double c22 = a * e - b * d;
    const double det = a * c00 + b * c01 + c * c02;
    if (det == 0.0) return false;
    const double adj[9] = {c00, c10, c20, c01, c11, c21, c02, c12, c22};
    for (int t = 0; t < 9; ++t) out[t] = adj[t] / det;
    return true;
  }
  const int w = 2 * n;
  std::vector<double> M((size_t)n * w, 0.0);
  for (int r = 0; r < n; ++r) {
    for (int c = 0; c < n; ++c) M[(size_t)r * w + c] = P[(size_t)r * n + c];
    M[(size_t)r * w + n + r] = 1.0;
  }
  for (int col = 0; col < n; ++col) {
    int piv = col;
    double best = std::fabs(M[(size_t)col * w + col]);
    for (int r = col + 1; r < n; ++r) {
      const double v = std::fabs(M[(size_t)r * w + col]);
      if (v > best) {
        best = v;
        piv = r;
      }
    }
    if (M[(size_t)piv * w + col] == 0.0) return false;
    if (piv != col)
      for (int c = 0; c < w; ++c) std::swap(M[(size_t)col * w + c], M[(size_t)piv * w + c]);
    const double p = M[(size_t)col * w + col];
    for (int c = 0; c < w; ++c) M[(size_t)col * w + c] = M[(size_t)col * w + c] / p;
    for (int r = 0; r < n; ++r) {
      if (r == col || M[(size_t)r * w + col] == 0.0) continue;
      const double f = M[(size_t)r * w + col];
      for (int c = 0; c < w; ++c)
        M[(size_t)r * w + c] = M[(size_t)r * w + c] - f * M[(size_t)col * w + c];
    }
  }
  for (int r = 0; r < n; ++r)
    for (int c = 0; c < n; ++c) out[(size_t)r * n + c] = M[(size_t)r * w + n + c];
  return true;
}

void build_lists(const fm_scheme& s, Lists& L) {
  const int gm = s.m, gk = s.k, gn = s.n, R = s.R;
  for (Side* side : {&L.a, &L.b, &L.w}) {
    side->off.assign(R + 1, 0);
    side->idx.clear();
    side->coef.clear();
  }
  // A coefficient is kept when its fp32 rounding (one rounding, to nearest
  // even) is nonzero.
  auto add = [](Side& sd, int idx, double c) {
    const float f = (float)c;
    if (f != 0.0f) {
      sd.idx.push_back(idx);
      sd.coef.push_back(f);
    }
  };
  for (int r = 0; r < R; ++r) {
    L.a.off[r] = (int32_t)L.a.idx.size();
    for (int i = 0; i < gm; ++i)
      for (int l = 0; l < gk; ++l) add(L.a, i * gk + l, s.U[(size_t)r * gm * gk + i * gk + l]);
    L.b.off[r] = (int32_t)L.b.idx.size();
    for (int l = 0; l < gk; ++l)
      for (int j = 0; j < gn; ++j) add(L.b, j * gk + l, s.V[(size_t)r * gk * gn + l * gn + j]);
    L.w.off[r] = (int32_t)L.w.idx.size();
    for (int i = 0; i < gm; ++i)
      for (int j = 0; j < gn; ++j) add(L.w, i * gn + j, s.W[(size_t)r * gm * gn + i * gn + j]);
  }
  L.a.off[R] = (int32_t)L.a.idx.size();
  L.b.off[R] = (int32_t)L.b.idx.size();
  L.w.off[R] = (int32_t)L.w.idx.size();
}

}  // namespace fm

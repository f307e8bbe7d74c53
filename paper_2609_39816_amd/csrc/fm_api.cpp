// C ABI of libfm (include/fm.h): argument checks, workspace layout, table
// upload and the launch sequence of the FP8 schedule.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <string>
#include <atomic>
#include <mutex>
#include <thread>
#include <vector>

#include "fm_internal.h"

namespace fm {

namespace {
thread_local std::string g_err;

constexpr size_t kAlign = 256;
size_t up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Pinned host staging buffer for table uploads and small downloads.  An
// event recorded after each upload guards reuse of the buffer.
struct Staging {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
thread_local Staging g_stage;

int stage_reserve(size_t n) {
  if (g_stage.pending) {
    if (int rc = hip_check(hipEventSynchronize(g_stage.ev), "hipEventSynchronize")) return rc;
    g_stage.pending = false;
  }
  if (n <= g_stage.cap) return FM_OK;
  if (g_stage.host) (void)hipHostFree(g_stage.host);
  g_stage.host = nullptr;
  g_stage.cap = 0;
  size_t cap = std::max<size_t>(n, 1 << 20);
  if (int rc = hip_check(hipHostMalloc(&g_stage.host, cap, hipHostMallocDefault), "hipHostMalloc"))
    return rc;
  g_stage.cap = cap;
  return FM_OK;
}

// Copies the host pieces into the staging buffer and uploads them with one
// asynchronous copy to `dst`.
int upload(void* dst, const std::vector<std::pair<const void*, size_t>>& pieces,
           const std::vector<size_t>& offsets, size_t total, hipStream_t st) {
  if (int rc = stage_reserve(total)) return rc;
  for (size_t i = 0; i < pieces.size(); ++i)
    std::memcpy((char*)g_stage.host + offsets[i], pieces[i].first, pieces[i].second);
  if (int rc = hip_check(hipMemcpyAsync(dst, g_stage.host, total, hipMemcpyHostToDevice, st),
                         "hipMemcpyAsync(H2D)"))
    return rc;
  if (!g_stage.ev)
    if (int rc = hip_check(hipEventCreateWithFlags(&g_stage.ev, hipEventDisableTiming),
                           "hipEventCreate"))
      return rc;
  if (int rc = hip_check(hipEventRecord(g_stage.ev, st), "hipEventRecord")) return rc;
  g_stage.pending = true;
  return FM_OK;
}

int download(void* host, const void* dev, size_t n, hipStream_t st) {
  if (int rc = stage_reserve(n)) return rc;
  if (int rc = hip_check(hipMemcpyAsync(g_stage.host, dev, n, hipMemcpyDeviceToHost, st),
                         "hipMemcpyAsync(D2H)"))
    return rc;
  if (int rc = hip_check(hipStreamSynchronize(st), "hipStreamSynchronize")) return rc;
  std::memcpy(host, g_stage.host, n);
  return FM_OK;
}

// Concatenated coefficient lists of G flattened schemes: offsets are
// absolute indices into the concatenated idx/coef arrays.  pat[side][g] is
// the pattern family of gauge g's list on that side (-1: none).
struct Tables {
  int G = 0, R = 0;
  Side s[3];
  std::vector<int> pat[3];
  std::vector<char> trie[2];  // per gauge: a sign variant of its family's base scheme
  std::vector<uint64_t> sgn[2];  // per gauge: its block signs (bit b: block b negated)
  std::vector<int> hpat;  // family of each gauge's H support (joint rounding only)
};

void append(Tables& T, const Lists& L, int R, const int nb[3]) {
  const Side* src[3] = {&L.a, &L.b, &L.w};
  for (int k = 0; k < 3; ++k) {
    Side& d = T.s[k];
    const int32_t base = (int32_t)d.idx.size();
    for (int r = 0; r <= R; ++r) d.off.push_back(base + src[k]->off[r]);
    d.idx.insert(d.idx.end(), src[k]->idx.begin(), src[k]->idx.end());
    d.coef.insert(d.coef.end(), src[k]->coef.begin(), src[k]->coef.end());
    T.pat[k].push_back(match_pattern(k, *src[k], R, nb[k]));
    if (k < 2) {
      uint64_t m = 0;
      const bool ok = block_signs(T.pat[k].back(), k, *src[k], nb[k], &m);
      T.trie[k].push_back(ok ? 1 : 0);
      T.sgn[k].push_back(ok ? m : 0);
    }
  }
  T.G += 1;
}

// 1 if every gauge of [g0, g0 + n) may use its family's prefix-shared chains
// on one side (A: 0, B: 1): every one is a sign variant of the base scheme.
int chunk_trie(const Tables& T, int side, int g0, int n) {
  for (int g = g0; g < g0 + n; ++g)
    if (!T.trie[side][g]) return 0;
  return 1;
}

// Pattern shared by gauges [g0, g0 + n) on one side, or -1.
int chunk_pattern(const Tables& T, int side, int g0, int n) {
  const int p = T.pat[side][g0];
  for (int g = g0 + 1; g < g0 + n; ++g)
    if (T.pat[side][g] != p) return -1;
  return p;
}

// Workspace layout for G gauges processed `chunk` at a time.
struct Layout {
  // *2: a second set of a chunk's maxima, scales and block products when the
  // orbit runs in several chunks (equal to the first set otherwise)
  size_t flags, bt, off[3], idx[3], coef[3], sg[2], amax, q, d, tq, sq, mprod, amax2, q2, d2, mprod2,
      partial, errsq, out3, arow, rowup, hg, hgc, hgp, total;
  int recon_nblk;
  bool two_sets() const { return mprod2 != mprod; }
  // the layout with set k in the first slots
  Layout set(int k) const {
    Layout o = *this;
    if (k) {
      o.amax = amax2;
      o.q = q2;
      o.d = d2;
      o.mprod = mprod2;
    }
    return o;
  }
};

// Scale-mode word: the granularity in the low byte, repair flags above it
// (FM_REPAIR_ROWS, FM_REPAIR_WEIGHTS; only with FM_SCALE_GROUP).
int base_mode(int scale_mode) { return scale_mode & 0xff; }
bool repair_rows(int scale_mode) { return (scale_mode & FM_REPAIR_ROWS) != 0; }
bool repair_weights(int scale_mode) { return (scale_mode & FM_REPAIR_WEIGHTS) != 0; }

// Scales per (gauge, product) on each side: 1, or one per block-sum row
// (A side, Mb) and per block-sum column (B side, Nb), or per group: (Kb/128)
// Mb on A's side and (Kb/128) (Nb/128) on B's.
int scales_a(const Geometry& g, int scale_mode) {
  const int m = base_mode(scale_mode);
  return m == FM_SCALE_ROWCOL ? g.Mb : m == FM_SCALE_GROUP ? g.Kb / 128 * g.Mb : 1;
}
int scales_b(const Geometry& g, int scale_mode) {
  const int m = base_mode(scale_mode);
  return m == FM_SCALE_ROWCOL ? g.Nb : m == FM_SCALE_GROUP ? g.Kb / 128 * (g.Nb / 128) : 1;
}
// Block shapes a scale mode needs (group scales: Kb, Nb multiples of 128,
// Mb of 4).
int scale_shape_ok(int Mb, int Nb, int Kb, int R, int scale_mode) {
  if (base_mode(scale_mode) == FM_SCALE_GROUP && (Kb % 128 || Nb % 128 || Mb % 4))
    return fail(FM_E_SHAPE, "group scales need Kb, Nb multiples of 128 and Mb of 4");
  // checked before any device work (the joint rounding keeps R-long state)
  if (repair_weights(scale_mode) && R > 64)
    return fail(FM_E_UNSUPPORTED, "joint rounding is built for at most 64 products");
  return FM_OK;
}

Layout make_layout(const Geometry& g, int G, int chunk, bool need_bt = true,
                   int scale_mode = FM_SCALE_TENSOR, bool two_sets = false) {
  Layout L{};
  const size_t R = (size_t)g.R;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += up(bytes);
    return at;
  };
  L.flags = take(kAlign);
  L.bt = take(need_bt ? (size_t)g.N * g.K * 4 : 0);
  const size_t nbk[3] = {(size_t)g.NBa(), (size_t)g.NBb(), (size_t)g.NC()};
  for (int k = 0; k < 3; ++k) {
    L.off[k] = take((size_t)G * (R + 1) * 4);
    L.idx[k] = take((size_t)G * R * nbk[k] * 4);
    L.coef[k] = take((size_t)G * R * nbk[k] * 4);
  }
  for (int k = 0; k < 2; ++k) L.sg[k] = take((size_t)G * 8);
  const size_t nsc = (size_t)chunk * R * (scales_a(g, scale_mode) + scales_b(g, scale_mode));
  L.amax = take(nsc * 4);
  L.q = take(nsc * 4);
  L.d = take(nsc * 4 + 16);  // whole 16-byte chunks for the kernels' scale loads
  L.tq = take((size_t)chunk * R * g.Mb * g.Kb);
  L.sq = take((size_t)chunk * R * g.Nb * g.Kb);
  L.mprod = take((size_t)chunk * R * g.Mb * g.Nb * 4);
  if (two_sets) {
    L.amax2 = take(nsc * 4);
    L.q2 = take(nsc * 4);
    L.d2 = take(nsc * 4 + 16);
    L.mprod2 = take((size_t)chunk * R * g.Mb * g.Nb * 4);
  } else {
    L.amax2 = L.amax;
    L.q2 = L.q;
    L.d2 = L.d;
    L.mprod2 = L.mprod;
  }
  ReconArgs ra{};
  ra.G = chunk;
  ra.gm = g.gm;
  ra.gn = g.gn;
  ra.Mb = g.Mb;
  ra.Nb = g.Nb;
  ra.N = g.N;
  L.recon_nblk = recon_blocks(ra);
  L.partial = take((size_t)chunk * L.recon_nblk * 8);
  L.errsq = take((size_t)G * 8);
  L.out3 = take(3 * 8);
  // repairs: A's rescaled rows and the row factors; every gauge's H
  L.arow = take(repair_rows(scale_mode) ? (size_t)g.M * g.K * 4 : 0);
  L.rowup = take(repair_rows(scale_mode) ? (size_t)g.M * 4 : 0);
  // every gauge's H in compressed rows: values, columns, row pointers
  L.hg = take(repair_weights(scale_mode) ? (size_t)G * R * R * 4 : 0);
  L.hgc = take(repair_weights(scale_mode) ? (size_t)G * R * R * 2 : 0);
  L.hgp = take(repair_weights(scale_mode) ? (size_t)G * (R + 1) * 4 : 0);
  L.total = o;
  return L;
}

// H_rs = <w_r, w_s> <u_r, u_s> for every gauge (the repair rules), from the
// fp32 coefficient lists: each inner product in float64 over ascending block
// index, their product rounded once to fp32.
// H of every gauge (G x R x R) and its support: the pairs whose products
// share a block of A and a block of C, where H can be nonzero (an entry of
// the support may still cancel to zero).
std::vector<float> repair_grams(const Tables& T, const Geometry& geo, std::vector<uint8_t>& sup) {
  const int R = T.R, nu = geo.NBa(), nw = geo.NC();
  std::vector<float> H((size_t)T.G * R * R);
  sup.assign((size_t)T.G * R * R, 0);
  std::vector<double> u((size_t)R * nu), w((size_t)R * nw);
  for (int g = 0; g < T.G; ++g) {
    std::fill(u.begin(), u.end(), 0.0);
    std::fill(w.begin(), w.end(), 0.0);
    for (int k : {0, 2}) {
      const Side& sd = T.s[k];
      std::vector<double>& dst = k == 0 ? u : w;
      const int n = k == 0 ? nu : nw;
      for (int r = 0; r < R; ++r)
        for (int e = sd.off[(size_t)g * (R + 1) + r]; e < sd.off[(size_t)g * (R + 1) + r + 1]; ++e)
          dst[(size_t)r * n + sd.idx[e]] = sd.coef[e];
    }
    for (int r = 0; r < R; ++r)
      for (int t = 0; t < R; ++t) {
        double uu = 0.0, ww = 0.0;
        bool su = false, sw = false;
        for (int i = 0; i < nu; ++i) {
          uu += u[(size_t)r * nu + i] * u[(size_t)t * nu + i];
          su |= u[(size_t)r * nu + i] != 0.0 && u[(size_t)t * nu + i] != 0.0;
        }
        for (int i = 0; i < nw; ++i) {
          ww += w[(size_t)r * nw + i] * w[(size_t)t * nw + i];
          sw |= w[(size_t)r * nw + i] != 0.0 && w[(size_t)t * nw + i] != 0.0;
        }
        H[((size_t)g * R + r) * R + t] = (float)(ww * uu);
        sup[((size_t)g * R + r) * R + t] = su && sw;
      }
  }
  return H;
}

// Repairs that act once per call: A's rows rescaled (returns the operand the
// formation reads and the row factors) and every gauge's H uploaded.
int prepare_repairs(const Geometry& geo, Tables& T, char* ws, const Layout& L,
                    int scale_mode, const float* A, const float*& Aform, const float*& rowup,
                    hipStream_t st) {
  Aform = A;
  rowup = nullptr;
  if (repair_rows(scale_mode)) {
    float* As = (float*)(ws + L.arow);
    float* up = (float*)(ws + L.rowup);
    if (int rc = launch_row_repair(A, geo.M, geo.K, As, up, st)) return rc;
    Aform = As;
    rowup = up;
  }
  if (repair_weights(scale_mode)) {
    // H in compressed rows over its support (an entry outside it is an
    // exact zero and is left out; one inside that cancels adds an exact
    // zero), so the rows of a family's gauges follow the family's H pattern
    std::vector<uint8_t> sup;
    const std::vector<float> H = repair_grams(T, geo, sup);
    const int R = T.R;
    std::vector<float> hv((size_t)T.G * R * R, 0.0f);
    std::vector<uint16_t> hc((size_t)T.G * R * R, 0);
    std::vector<int32_t> hp((size_t)T.G * (R + 1), 0);
    T.hpat.assign(T.G, -1);
    for (int g = 0; g < T.G; ++g) {
      int n = 0;
      for (int r = 0; r < R; ++r) {
        hp[(size_t)g * (R + 1) + r] = n;
        for (int t = 0; t < R; ++t) {
          if (!sup[((size_t)g * R + r) * R + t]) continue;
          hv[(size_t)g * R * R + n] = H[((size_t)g * R + r) * R + t];
          hc[(size_t)g * R * R + n] = (uint16_t)t;
          ++n;
        }
      }
      hp[(size_t)g * (R + 1) + R] = n;
      T.hpat[g] = match_h_pattern(hp.data() + (size_t)g * (R + 1), hc.data() + (size_t)g * R * R, R);
    }
    // the three tables are adjacent in the workspace: one staged copy
    if (int rc = upload(ws + L.hg,
                        {{hv.data(), hv.size() * 4}, {hc.data(), hc.size() * 2},
                         {hp.data(), hp.size() * 4}},
                        {0, L.hgc - L.hg, L.hgp - L.hg}, L.hgp - L.hg + hp.size() * 4, st))
      return rc;
  }
  return FM_OK;
}

int check_geometry(const fm_scheme* s, int levels, int M, int N, int K, Geometry& g) {
  if (!s) return fail(FM_E_ARG, "null scheme");
  if (levels < 1 || levels > 8) return fail(FM_E_ARG, "levels must be in [1, 8]");
  if (M < 1 || N < 1 || K < 1) return fail(FM_E_ARG, "M, N, K must be positive");
  long long gm = 1, gk = 1, gn = 1, R = 1;
  for (int l = 0; l < levels; ++l) {
    gm *= s->m;
    gk *= s->k;
    gn *= s->n;
    R *= s->R;
    if (gm > 64 || gk > 64 || gn > 64 || R > (1 << 20))
      return fail(FM_E_UNSUPPORTED, "flattened scheme too large");
  }
  g.gm = (int)gm;
  g.gk = (int)gk;
  g.gn = (int)gn;
  g.R = (int)R;
  g.M = M;
  g.N = N;
  g.K = K;
  if (M % gm || N % gn || K % gk)
    return fail(FM_E_SHAPE, "M, N, K must be multiples of the flattened grid (" +
                                std::to_string(gm) + ", " + std::to_string(gn) + ", " +
                                std::to_string(gk) + ")");
  g.Mb = M / (int)gm;
  g.Nb = N / (int)gn;
  g.Kb = K / (int)gk;
  if (g.Kb % 16) return fail(FM_E_SHAPE, "inner block length K/k^L must be a multiple of 16");
  if ((long long)M * K >= (1LL << 40) || (long long)K * N >= (1LL << 40) ||
      (long long)M * N >= (1LL << 40))
    return fail(FM_E_SHAPE, "operand too large");
  if (g.NBa() > 64 || g.NBb() > 64 || g.NC() > 64)
    return fail(FM_E_UNSUPPORTED, "more than 64 blocks per operand");
  return FM_OK;
}

int check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(FM_E_WORKSPACE, "null workspace");
  if ((uintptr_t)ws % kAlign) return fail(FM_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return fail(FM_E_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, got " +
                                    std::to_string(ws_bytes));
  return FM_OK;
}

// Appends the lists of gauges [g_from, g_to) to T.
int extend_tables(Tables& T, const fm_scheme* const* schemes, int g_from, int g_to, int levels,
                  const Geometry& geo) {
  T.R = geo.R;
  for (int g = g_from; g < g_to; ++g) {
    const fm_scheme* s = schemes[g];
    if (!s) return fail(FM_E_ARG, "null scheme in orbit");
    // one level: the scheme itself (no copy)
    fm_scheme powered;
    if (levels > 1) powered = power(*s, levels);
    const fm_scheme& flat = levels > 1 ? powered : *s;
    if (flat.m != geo.gm || flat.k != geo.gk || flat.n != geo.gn || flat.R != geo.R)
      return fail(FM_E_MISMATCH, "schemes of one orbit must share grid and rank");
    Lists L;
    build_lists(flat, L);
    const int nb[3] = {geo.NBa(), geo.NBb(), geo.NC()};
    append(T, L, geo.R, nb);
  }
  return FM_OK;
}

// Uploads the tables of gauges [g_from, g_to) (already in T) to their
// places in the workspace: one asynchronous copy per table region.  The
// staging buffer must hold them (stage_reserve).
int upload_table_range(const Tables& T, char* ws, const Layout& L, int g_from, int g_to,
                       hipStream_t st) {
  const size_t R1 = (size_t)T.R + 1;
  std::vector<std::pair<const void*, size_t>> pieces;
  std::vector<size_t> dst;
  for (int k = 0; k < 3; ++k) {
    const Side& sd = T.s[k];
    const size_t e0 = (size_t)sd.off[(size_t)g_from * R1];
    const size_t e1 = (size_t)sd.off[(size_t)(g_to - 1) * R1 + T.R];
    pieces.push_back({sd.off.data() + (size_t)g_from * R1, (size_t)(g_to - g_from) * R1 * 4});
    dst.push_back(L.off[k] + (size_t)g_from * R1 * 4);
    pieces.push_back({sd.idx.data() + e0, (e1 - e0) * 4});
    dst.push_back(L.idx[k] + e0 * 4);
    pieces.push_back({sd.coef.data() + e0, (e1 - e0) * 4});
    dst.push_back(L.coef[k] + e0 * 4);
  }
  for (int k = 0; k < 2; ++k) {
    pieces.push_back({T.sgn[k].data() + g_from, (size_t)(g_to - g_from) * 8});
    dst.push_back(L.sg[k] + (size_t)g_from * 8);
  }
  size_t total = 0;
  for (auto& p : pieces) total += p.second;
  if (int rc = stage_reserve(total)) return rc;
  size_t at = 0;
  for (size_t i = 0; i < pieces.size(); ++i) {
    if (!pieces[i].second) continue;
    std::memcpy((char*)g_stage.host + at, pieces[i].first, pieces[i].second);
    if (int rc = hip_check(hipMemcpyAsync(ws + dst[i], (char*)g_stage.host + at, pieces[i].second,
                                          hipMemcpyHostToDevice, st),
                           "hipMemcpyAsync(H2D)"))
      return rc;
    at += pieces[i].second;
  }
  if (!g_stage.ev)
    if (int rc = hip_check(hipEventCreateWithFlags(&g_stage.ev, hipEventDisableTiming),
                           "hipEventCreate"))
      return rc;
  if (int rc = hip_check(hipEventRecord(g_stage.ev, st), "hipEventRecord")) return rc;
  g_stage.pending = true;
  return FM_OK;
}

Tables make_tables(const fm_scheme* const* schemes, int G, int levels, const Geometry& geo,
                   int& rc) {
  Tables T;
  T.R = geo.R;
  rc = FM_OK;
  for (int g = 0; g < G; ++g) {
    const fm_scheme* s = schemes[g];
    if (!s) {
      rc = fail(FM_E_ARG, "null scheme in orbit");
      return T;
    }
    fm_scheme flat = power(*s, levels);
    if (flat.m != geo.gm || flat.k != geo.gk || flat.n != geo.gn || flat.R != geo.R) {
      rc = fail(FM_E_MISMATCH, "schemes of one orbit must share grid and rank");
      return T;
    }
    Lists L;
    build_lists(flat, L);
    const int nb[3] = {geo.NBa(), geo.NBb(), geo.NC()};
    append(T, L, geo.R, nb);
  }
  return T;
}

int upload_tables(const Tables& T, char* ws, const Layout& L, hipStream_t st) {
  // one contiguous region from the first table to the end of the last
  const size_t base = L.off[0];
  const size_t total = L.sg[1] + T.sgn[1].size() * 8 - base;
  std::vector<std::pair<const void*, size_t>> pieces;
  std::vector<size_t> offs;
  for (int k = 0; k < 3; ++k) {
    pieces.push_back({T.s[k].off.data(), T.s[k].off.size() * 4});
    offs.push_back(L.off[k] - base);
    pieces.push_back({T.s[k].idx.data(), T.s[k].idx.size() * 4});
    offs.push_back(L.idx[k] - base);
    pieces.push_back({T.s[k].coef.data(), T.s[k].coef.size() * 4});
    offs.push_back(L.coef[k] - base);
  }
  for (int k = 0; k < 2; ++k) {
    pieces.push_back({T.sgn[k].data(), T.sgn[k].size() * 8});
    offs.push_back(L.sg[k] - base);
  }
  return upload(ws + base, pieces, offs, total, st);
}

// The prefix-shared chains for gauges [g0, g0 + n) of one side: the flag,
// and the gauges' block-sign masks when it is set.
void set_trie(FormArgs& f, const Tables& T, char* ws, const Layout& L, int side, int g0, int n) {
  f.trie = chunk_trie(T, side, g0, n);
  f.sgn = f.trie ? (const uint64_t*)(ws + L.sg[side]) + g0 : nullptr;
}

// Formation arguments of both sides of the gauges [g0, g0 + n) with one
// scale per block-sum tensor, maxima and scales in the first set of L.
void tensor_form_args(const Geometry& geo, const float* A, const float* Bt, char* ws,
                      const Layout& L, int g0, int n, int fmt, uint8_t* Tq, uint8_t* Sq,
                      FormArgs& fa, FormArgs& fb) {
  const int R = geo.R;
  const size_t na = (size_t)n * R;
  uint32_t* amax = (uint32_t*)(ws + L.amax);
  float* q = (float*)(ws + L.q);
  auto off = [&](int k) { return (const int32_t*)(ws + L.off[k]) + (size_t)g0 * (R + 1); };
  auto idx = [&](int k) { return (const int32_t*)(ws + L.idx[k]); };
  auto coef = [&](int k) { return (const float*)(ws + L.coef[k]); };
  fa = FormArgs{A,    geo.M, geo.K, geo.gm, geo.gk, geo.Mb, geo.Kb, off(0), idx(0), coef(0), R, n,
                amax, q,     Tq,    fmt,    0,      1};
  fb = FormArgs{Bt,       geo.N,    geo.K, geo.gn, geo.gk, geo.Nb, geo.Kb, off(1), idx(1), coef(1),
                R,        n,        amax + na, q + na, Sq, fmt, 0, 1};
}

// Per-tensor scales of an orbit in several chunks: the FP8 codes of chunk c
// and the maxima of chunk c + 1 are formed in one pass per side (the merged
// kernel, when both chunks are of one kernel family; otherwise the two passes
// separately), then the scales of chunk c + 1 (the other set of L).  The
// maxima and scales of chunk 0 are formed first, by the caller.
int form_codes_and_next_maxima(const Geometry& geo, const float* A, const float* Bt, char* ws,
                               const Layout& L, const Tables& T, int c, int g0, int n, int n1,
                               int fmt, uint8_t* Tq, uint8_t* Sq, hipStream_t st) {
  FormArgs qa, qb, ma, mb;
  tensor_form_args(geo, A, Bt, ws, L.set(c & 1), g0, n, fmt, Tq, Sq, qa, qb);
  set_trie(qa, T, ws, L, 0, g0, n);
  set_trie(qb, T, ws, L, 1, g0, n);
  const Layout Ln = L.set((c + 1) & 1);
  if (n1 > 0) {
    tensor_form_args(geo, A, Bt, ws, Ln, g0 + n, n1, fmt, Tq, Sq, ma, mb);
    set_trie(ma, T, ws, L, 0, g0 + n, n1);
    set_trie(mb, T, ws, L, 1, g0 + n, n1);
    if (int rc = launch_fill_u32(ma.amax, (size_t)2 * n1 * geo.R, 0u, st)) return rc;
  }
  for (int side = 0; side < 2; ++side) {
    const int pq = chunk_pattern(T, side, g0, n);
    const int pm = n1 > 0 ? chunk_pattern(T, side, g0 + n, n1) : -1;
    const FormArgs& aq = side ? qb : qa;
    const FormArgs& am = side ? mb : ma;
    timing_begin(T_FORM_QUANT, st);
    const bool merge = n1 > 0 && pq >= 0 && pq == pm;
    int rc = merge ? launch_form_merged(aq, am, pq, side, st) : 1;
    const bool merged = merge && rc != 1;
    if (!merged) rc = launch_form(aq, 1, pq, side, st);
    if (rc) return rc;
    timing_end(T_FORM_QUANT, st);
    if (n1 > 0 && !merged) {
      timing_begin(T_FORM_AMAX, st);
      if ((rc = launch_form(am, 0, pm, side, st))) return rc;
      timing_end(T_FORM_AMAX, st);
    }
  }
  if (n1 > 0)
    return launch_scales(ma.amax, (float*)(ws + Ln.q), (float*)(ws + Ln.d), 2 * n1 * geo.R, fmt,
                         (uint32_t*)(ws + L.flags), st);
  return FM_OK;
}

// Operand formation for gauges [g0, g0 + n) of the uploaded tables.
int form_chunk(const Geometry& geo, const float* A, const float* Bt, char* ws, const Layout& L,
               const Tables& T, int g0, int n, int fmt, int scale_mode, uint8_t* Tq, uint8_t* Sq,
               float* dT, float* dS, hipStream_t st) {
  const int R = geo.R;
  // finer granularities fold their maxima into global memory by group:
  // rows (per-row form), or 1 x 128 groups on A's side and bf16-rounded
  // 128 x 128 blocks on B's (group schedule)
  const int mode = base_mode(scale_mode);
  const int per_row = mode == FM_SCALE_TENSOR ? 0 : 1;
  const size_t na = (size_t)n * R * scales_a(geo, scale_mode);
  const size_t nb = (size_t)n * R * scales_b(geo, scale_mode);
  uint32_t* amax = (uint32_t*)(ws + L.amax);
  float* q = (float*)(ws + L.q);
  float* dd = (float*)(ws + L.d);
  auto off = [&](int k) { return (const int32_t*)(ws + L.off[k]) + (size_t)g0 * (R + 1); };
  auto idx = [&](int k) { return (const int32_t*)(ws + L.idx[k]); };
  auto coef = [&](int k) { return (const float*)(ws + L.coef[k]); };
  const int pa = chunk_pattern(T, 0, g0, n), pb = chunk_pattern(T, 1, g0, n);
  FormArgs fa{A,    geo.M, geo.K, geo.gm, geo.gk, geo.Mb, geo.Kb, off(0), idx(0), coef(0), R, n,
              amax, q,     Tq,    fmt,    per_row, mode == FM_SCALE_GROUP ? 2 : 1};
  FormArgs fb{Bt, geo.N, geo.K, geo.gn, geo.gk, geo.Nb, geo.Kb, off(1), idx(1), coef(1), R, n,
              amax + na, q + na, Sq, fmt, per_row, mode == FM_SCALE_GROUP ? 3 : 1};
  set_trie(fa, T, ws, L, 0, g0, n);
  set_trie(fb, T, ws, L, 1, g0, n);
  if (int rc = launch_fill_u32(amax, na + nb, 0u, st)) return rc;
  for (int side = 0; side < 2; ++side) {
    timing_begin(T_FORM_AMAX, st);
    if (int rc = launch_form(side ? fb : fa, 0, side ? pb : pa, side, st)) return rc;
    timing_end(T_FORM_AMAX, st);
  }
  if (int rc = launch_scales(amax, q, dd, (int)(na + nb), fmt, (uint32_t*)(ws + L.flags), st))
    return rc;
  // with joint rounding B's codes come from it alone (it writes every one)
  const int quant_sides = repair_weights(scale_mode) ? 1 : 2;
  for (int side = 0; side < quant_sides; ++side) {
    timing_begin(T_FORM_QUANT, st);
    if (int rc = launch_form(side ? fb : fa, 1, side ? pb : pa, side, st)) return rc;
    timing_end(T_FORM_QUANT, st);
  }
  if (repair_weights(scale_mode)) {
    // the family kernel needs B's lists and H's support both of its family
    int ph = T.hpat.empty() ? -1 : T.hpat[g0];
    for (int g = g0 + 1; g < g0 + n && ph >= 0; ++g)
      if (T.hpat[g] != ph) ph = -1;
    timing_begin(T_FORM_QUANT, st);
    if (int rc = launch_joint_round(fb, q + na, dd + na,
                                    (const float*)(ws + L.hg) + (size_t)g0 * R * R,
                                    (const uint16_t*)(ws + L.hgc) + (size_t)g0 * R * R,
                                    (const int32_t*)(ws + L.hgp) + (size_t)g0 * (R + 1),
                                    pb >= 0 && pb == ph ? pb : -1, st))
      return rc;
    timing_end(T_FORM_QUANT, st);
  }
  if (dT)
    if (int rc = hip_check(hipMemcpyAsync(dT, dd, na * 4, hipMemcpyDeviceToDevice, st),
                           "hipMemcpyAsync(dT)"))
      return rc;
  if (dS)
    if (int rc = hip_check(hipMemcpyAsync(dS, dd + na, nb * 4, hipMemcpyDeviceToDevice, st),
                           "hipMemcpyAsync(dS)"))
      return rc;
  return FM_OK;
}

// Two-stream schedule of an orbit in several chunks: the caller's stream
// forms operands and runs the block products; a second stream of the same
// (default) priority reconstructs each chunk from its product buffer, so
// that work runs beside the next chunk's formation.  Events order the two:
// a chunk's reconstruction waits for its products, products of chunk c wait
// until chunk c - 1 has been reconstructed, and the caller's stream waits
// for every reconstruction at the end (also on an early return, so no work
// is left running on the workspace).
hipStream_t side_stream(int& rc) {
  static std::mutex mu;
  static hipStream_t streams[64] = {};
  int dev = 0;
  if ((rc = hip_check(hipGetDevice(&dev), "hipGetDevice"))) return nullptr;
  if (dev < 0 || dev >= 64) {
    rc = fail(FM_E_HIP, "device index out of range");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!streams[dev] &&
      (rc = hip_check(hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking),
                      "hipStreamCreateWithFlags")))
    return nullptr;
  return streams[dev];
}

struct Pipeline {
  bool on = false;
  hipStream_t main = nullptr, side = nullptr;
  hipEvent_t made[2] = {}, read[2] = {}, done = nullptr;

  int open(hipStream_t st) {
    int rc = FM_OK;
    main = st;
    side = side_stream(rc);
    if (rc) return rc;
    for (hipEvent_t* e : {&made[0], &made[1], &read[0], &read[1], &done})
      if ((rc = hip_check(hipEventCreateWithFlags(e, hipEventDisableTiming), "hipEventCreate")))
        return rc;
    on = true;
    return FM_OK;
  }
  // products of the buffer are written: the side stream takes over
  int hand_over(int buf, hipStream_t& rs) {
    if (int rc = hip_check(hipEventRecord(made[buf], main), "hipEventRecord")) return rc;
    if (int rc = hip_check(hipStreamWaitEvent(side, made[buf], 0), "hipStreamWaitEvent")) return rc;
    rs = side;
    return FM_OK;
  }
  int reconstructed(int buf) {
    return hip_check(hipEventRecord(read[buf], side), "hipEventRecord");
  }
  int wait_reconstructed(int buf) {
    if (!on) return FM_OK;
    return hip_check(hipStreamWaitEvent(main, read[buf], 0), "hipStreamWaitEvent");
  }
  int join() {
    if (!on) return FM_OK;
    on = false;
    if (int rc = hip_check(hipEventRecord(done, side), "hipEventRecord")) return rc;
    return hip_check(hipStreamWaitEvent(main, done, 0), "hipStreamWaitEvent");
  }
  ~Pipeline() {
    if (on) {
      (void)hipEventRecord(done, side);
      (void)hipStreamWaitEvent(main, done, 0);
      (void)hipStreamSynchronize(side);
    }
    for (hipEvent_t e : {made[0], made[1], read[0], read[1], done})
      if (e) (void)hipEventDestroy(e);
  }
};

ReconArgs recon_args(const Geometry& geo, const char* ws, const Layout& L, int g0, int n,
                     const float* Mp, float* C, const double* Cref) {
  ReconArgs ra{Mp,
               (const int32_t*)(ws + L.off[2]) + (size_t)g0 * (geo.R + 1),
               (const int32_t*)(ws + L.idx[2]),
               (const float*)(ws + L.coef[2]),
               geo.R,
               n,
               geo.gm,
               geo.gn,
               geo.Mb,
               geo.Nb,
               geo.N,
               C,
               Cref,
               (double*)(ws + L.partial)};
  return ra;
}

int fmt_ok(int fmt) { return fmt == FM_E4M3 || fmt == FM_E5M2; }

fm_scheme* clone(const fm_scheme& s) {
  try {
    return new fm_scheme(s);
  } catch (...) {
    return nullptr;
  }
}
fm_scheme* clone(fm_scheme&& s) {
  try {
    return new fm_scheme(std::move(s));
  } catch (...) {
    return nullptr;
  }
}

}  // namespace

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

// An exception inside an exported call (a host allocation that failed, or a
// container asked for more than it can hold) ends the call with FM_E_NOMEM:
// every exported function is a function-try-block that returns this value
// (0 or "" for the size and name queries).  Setting the message may itself
// fail; the message is then left empty.
int host_failure() noexcept {
  try {
    g_err = "host allocation failed";
  } catch (...) {
    g_err.clear();
  }
  return FM_E_NOMEM;
}

// ----------------------------------------------------------- kernel timing
namespace {
const char* const kTimedNames[T_COUNT] = {"form_amax", "form_quant", "block_gemm", "recon",
                                          "reference"};
struct TimingRec {
  int cls;
  hipEvent_t start, stop;
};
struct Timing {
  bool on = false;
  std::vector<TimingRec> recs;
  std::vector<hipEvent_t> pool;
  int open_cls = -1;
  hipEvent_t open_start = nullptr;
} g_timing;

hipEvent_t timing_event() {
  if (!g_timing.pool.empty()) {
    hipEvent_t e = g_timing.pool.back();
    g_timing.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

void timing_begin(int cls, hipStream_t st) {
  if (!g_timing.on) return;
  g_timing.open_cls = cls;
  g_timing.open_start = timing_event();
  if (g_timing.open_start) (void)hipEventRecord(g_timing.open_start, st);
}

void timing_end(int cls, hipStream_t st) {
  if (!g_timing.on || g_timing.open_cls != cls || !g_timing.open_start) return;
  hipEvent_t stop = timing_event();
  if (!stop) return;
  (void)hipEventRecord(stop, st);
  g_timing.recs.push_back({cls, g_timing.open_start, stop});
  g_timing.open_cls = -1;
  g_timing.open_start = nullptr;
}

void clear_error() { g_err.clear(); }

int hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return FM_OK;
  return fail(FM_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace fm

using namespace fm;

extern "C" {

const char* fm_strerror(int code) {
  switch (code) {
    case FM_OK: return "ok";
    case FM_E_ARG: return "invalid argument";
    case FM_E_SHAPE: return "shape not supported by the block grid";
    case FM_E_BRENT: return "coefficients do not compute the matrix product";
    case FM_E_SINGULAR: return "singular gauge matrix";
    case FM_E_NONFINITE: return "non-finite value in a block sum";
    case FM_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case FM_E_HIP: return "HIP runtime error";
    case FM_E_MISMATCH: return "schemes of one orbit differ in shape";
    case FM_E_NOMEM: return "host allocation failed";
    case FM_E_UNSUPPORTED: return "unsupported scheme size";
    case FM_E_RANGE: return "a block sum of integer codes left int8";
    case FM_E_UNCERTIFIED: return "not certified: the conditions of Prop. 1 fail";
    default: return "unknown error";
  }
}

const char* fm_last_error(void) { return g_err.c_str(); }

const char* fm_version(void) { return "libfm 0.1 (gfx950)"; }

int fm_scheme_load(const double* U, const double* V, const double* W, int m, int n, int k, int R,
                   fm_scheme** out) try {
  clear_error();
  if (!U || !V || !W || !out) return fail(FM_E_ARG, "null pointer");
  *out = nullptr;
  if (m < 1 || n < 1 || k < 1 || m > 16 || n > 16 || k > 16 || R < 1 || R > 4096)
    return fail(FM_E_ARG, "sizes out of range");
  fm_scheme s;
  s.m = m;
  s.n = n;
  s.k = k;
  s.R = R;
  s.U.assign(U, U + (size_t)R * m * k);
  s.V.assign(V, V + (size_t)R * k * n);
  s.W.assign(W, W + (size_t)R * m * n);
  for (double x : s.U)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite coefficient");
  for (double x : s.V)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite coefficient");
  for (double x : s.W)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite coefficient");
  const double res = brent_residual(s);
  if (!(res <= 1e-9))
    return fail(FM_E_BRENT, "Brent residual " + std::to_string(res) + " exceeds 1e-9");
  *out = clone(s);
  return *out ? FM_OK : fail(FM_E_NOMEM, "out of host memory");
} catch (...) {
  return host_failure();
}

static int gauge_one(const fm_scheme* s, const double* P, const double* Q, const double* S,
                     fm_scheme** out) {
  *out = nullptr;
  const int m = s->m, k = s->k, n = s->n;
  std::vector<double> Pm(P, P + (size_t)m * m), Qm(Q, Q + (size_t)k * k), Sm(S, S + (size_t)n * n);
  for (double x : Pm)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite gauge entry");
  for (double x : Qm)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite gauge entry");
  for (double x : Sm)
    if (!std::isfinite(x)) return fail(FM_E_ARG, "non-finite gauge entry");
  std::vector<double> Pi, Qi, Si;
  if (!invert(Pm, m, Pi) || !invert(Qm, k, Qi) || !invert(Sm, n, Si))
    return fail(FM_E_SINGULAR, "gauge matrix is singular");
  fm_scheme g;
  g.m = m;
  g.n = n;
  g.k = k;
  g.R = s->R;
  g.U.assign(s->U.size(), 0.0);
  g.V.assign(s->V.size(), 0.0);
  g.W.assign(s->W.size(), 0.0);
  auto diagonal = [](const std::vector<double>& X, int n) {
    for (int a = 0; a < n; ++a)
      for (int b = 0; b < n; ++b)
        if (a != b && X[(size_t)a * n + b] != 0.0) return false;
    return true;
  };
  if (diagonal(Pm, m) && diagonal(Qm, k) && diagonal(Sm, n)) {
    // Each sum of the general formula below has one nonzero term, and the
    // accumulator starts at +0, so the result is exactly
    // (P_aa u_ab) Q_bb, (Qi_aa v_ab) S_bb, (Pi_aa w_ab) Si_bb.
    for (int r = 0; r < s->R; ++r) {
      for (int a = 0; a < m; ++a)
        for (int b = 0; b < k; ++b) {
          const size_t o = (size_t)r * m * k + (size_t)a * k + b;
          g.U[o] = (Pm[(size_t)a * m + a] * s->U[o]) * Qm[(size_t)b * k + b];
        }
      for (int a = 0; a < k; ++a)
        for (int b = 0; b < n; ++b) {
          const size_t o = (size_t)r * k * n + (size_t)a * n + b;
          g.V[o] = (Qi[(size_t)a * k + a] * s->V[o]) * Sm[(size_t)b * n + b];
        }
      for (int a = 0; a < m; ++a)
        for (int b = 0; b < n; ++b) {
          const size_t o = (size_t)r * m * n + (size_t)a * n + b;
          g.W[o] = (Pi[(size_t)a * m + a] * s->W[o]) * Si[(size_t)b * n + b];
        }
    }
    *out = clone(std::move(g));
    return *out ? FM_OK : fail(FM_E_NOMEM, "out of host memory");
  }
  // Terms with an exactly zero factor are skipped: the accumulator starts at
  // +0 and can never become -0, so adding a zero term would leave it
  // unchanged anyway (inputs are finite); the results are bit-identical to
  // the plain sums and diagonal gauges cost a quarter of the work.
  std::vector<double> t1, t2;
  for (int r = 0; r < s->R; ++r) {
    // U'_r = (P^T U_r) Q^T
    const double* u = &s->U[(size_t)r * m * k];
    t1.assign((size_t)m * k, 0.0);
    for (int a = 0; a < m; ++a)
      for (int b = 0; b < k; ++b) {
        double acc = 0.0;
        for (int c = 0; c < m; ++c) if (Pm[(size_t)c * m + a] != 0.0 && u[(size_t)c * k + b] != 0.0) acc = acc + Pm[(size_t)c * m + a] * u[(size_t)c * k + b];
        t1[(size_t)a * k + b] = acc;
      }
    for (int a = 0; a < m; ++a)
      for (int b = 0; b < k; ++b) {
        double acc = 0.0;
        for (int c = 0; c < k; ++c) if (t1[(size_t)a * k + c] != 0.0 && Qm[(size_t)b * k + c] != 0.0) acc = acc + t1[(size_t)a * k + c] * Qm[(size_t)b * k + c];
        g.U[(size_t)r * m * k + (size_t)a * k + b] = acc;
      }
    // V'_r = (Q^-T V_r) S^T
    const double* v = &s->V[(size_t)r * k * n];
    t2.assign((size_t)k * n, 0.0);
    for (int a = 0; a < k; ++a)
      for (int b = 0; b < n; ++b) {
        double acc = 0.0;
        for (int c = 0; c < k; ++c) if (Qi[(size_t)c * k + a] != 0.0 && v[(size_t)c * n + b] != 0.0) acc = acc + Qi[(size_t)c * k + a] * v[(size_t)c * n + b];
        t2[(size_t)a * n + b] = acc;
      }
    for (int a = 0; a < k; ++a)
      for (int b = 0; b < n; ++b) {
        double acc = 0.0;
        for (int c = 0; c < n; ++c) if (t2[(size_t)a * n + c] != 0.0 && Sm[(size_t)b * n + c] != 0.0) acc = acc + t2[(size_t)a * n + c] * Sm[(size_t)b * n + c];
        g.V[(size_t)r * k * n + (size_t)a * n + b] = acc;
      }
    // W'_r = (P^-1 W_r) S^-1
    const double* w = &s->W[(size_t)r * m * n];
    t1.assign((size_t)m * n, 0.0);
    for (int a = 0; a < m; ++a)
      for (int b = 0; b < n; ++b) {
        double acc = 0.0;
        for (int c = 0; c < m; ++c) if (Pi[(size_t)a * m + c] != 0.0 && w[(size_t)c * n + b] != 0.0) acc = acc + Pi[(size_t)a * m + c] * w[(size_t)c * n + b];
        t1[(size_t)a * n + b] = acc;
      }
    for (int a = 0; a < m; ++a)
      for (int b = 0; b < n; ++b) {
        double acc = 0.0;
        for (int c = 0; c < n; ++c) if (t1[(size_t)a * n + c] != 0.0 && Si[(size_t)c * n + b] != 0.0) acc = acc + t1[(size_t)a * n + c] * Si[(size_t)c * n + b];
        g.W[(size_t)r * m * n + (size_t)a * n + b] = acc;
      }
  }
  // The base scheme passed the Brent check at load; the gauged scheme then
  // computes AB exactly whenever the inverses are inverses.  Check that
  // (relative to the matrices' magnitudes) instead of the O(R (mkn)^2) Brent
  // tensor, which dominated the cost of gauging an orbit.
  auto inverse_ok = [](const std::vector<double>& X, const std::vector<double>& Xi, int n) {
    double mx = 0, mi = 0;
    for (double v : X) mx = std::max(mx, std::fabs(v));
    for (double v : Xi) mi = std::max(mi, std::fabs(v));
    for (int a = 0; a < n; ++a)
      for (int b = 0; b < n; ++b) {
        double acc = 0.0;
        for (int c = 0; c < n; ++c) acc = acc + X[(size_t)a * n + c] * Xi[(size_t)c * n + b];
        if (!(std::fabs(acc - (a == b ? 1.0 : 0.0)) <= 1e-12 * std::max(1.0, n * mx * mi)))
          return false;
      }
    return true;
  };
  if (!inverse_ok(Pm, Pi, m) || !inverse_ok(Qm, Qi, k) || !inverse_ok(Sm, Si, n))
    return fail(FM_E_SINGULAR, "gauge matrix is too ill-conditioned to invert accurately");
  *out = clone(std::move(g));
  return *out ? FM_OK : fail(FM_E_NOMEM, "out of host memory");
}

int fm_gauge_apply(const fm_scheme* s, const double* P, const double* Q, const double* S,
                   fm_scheme** out) try {
  clear_error();
  if (!s || !P || !Q || !S || !out) return fail(FM_E_ARG, "null pointer");
  return gauge_one(s, P, Q, S, out);
} catch (...) {
  return host_failure();
}

int fm_gauge_apply_batch(const fm_scheme* s, int G, const double* P, const double* Q,
                         const double* S, fm_scheme** out) try {
  clear_error();
  if (!s || !P || !Q || !S || !out) return fail(FM_E_ARG, "null pointer");
  if (G < 0) return fail(FM_E_ARG, "G must be non-negative");
  const size_t mm = (size_t)s->m * s->m, kk = (size_t)s->k * s->k, nn = (size_t)s->n * s->n;
  for (int g = 0; g < G; ++g) out[g] = nullptr;
  // gauges are independent: up to 16 host threads take them in turn (each
  // gauge of a three-level orbit is about half a millisecond of arithmetic
  // and copying); a failure is reported for the first failing gauge, by
  // applying it again on the calling thread (errors are per thread)
  std::vector<int> rcs((size_t)G, 0);
  std::atomic<int> next{0};
  auto work = [&] {
    for (;;) {
      const int g = next.fetch_add(1);
      if (g >= G) break;
      // no exception may leave a worker thread (that would end the process)
      try {
        rcs[g] = gauge_one(s, P + g * mm, Q + g * kk, S + g * nn, &out[g]);
      } catch (...) {
        rcs[g] = FM_E_NOMEM;
      }
    }
  };
  const long long per_gauge = (long long)s->R * (s->m * s->k + s->k * s->n + s->m * s->n);
  const int hw = std::max(1, (int)std::thread::hardware_concurrency());
  const int nt = per_gauge * G < (1 << 16) ? 1 : std::min(std::min(16, hw), G);
  std::vector<std::thread> pool;
  try {
    for (int i = 1; i < nt; ++i) pool.emplace_back(work);
  } catch (...) {
    // fewer threads: the calling thread takes the rest
  }
  work();
  for (auto& th : pool) th.join();
  for (int g = 0; g < G; ++g) {
    if (rcs[g]) {
      for (int h = 0; h < G; ++h) {
        fm_scheme_free(out[h]);
        out[h] = nullptr;
      }
      if (rcs[g] == FM_E_NOMEM) return fail(FM_E_NOMEM, "out of host memory");
      fm_scheme* again = nullptr;
      int rc;
      try {
        rc = gauge_one(s, P + g * mm, Q + g * kk, S + g * nn, &again);
      } catch (...) {
        rc = fail(FM_E_NOMEM, "out of host memory");
      }
      fm_scheme_free(again);
      return rc ? rc : rcs[g];
    }
  }
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_scheme_kron(const fm_scheme* s, int levels, fm_scheme** out) try {
  clear_error();
  if (!s || !out) return fail(FM_E_ARG, "null pointer");
  *out = nullptr;
  if (levels < 1 || levels > 8) return fail(FM_E_ARG, "levels must be in [1, 8]");
  long long R = 1, m = 1, n = 1, k = 1;
  for (int l = 0; l < levels; ++l) {
    R *= s->R;
    m *= s->m;
    n *= s->n;
    k *= s->k;
  }
  if (R > (1 << 20) || m * k * R > (1LL << 28) || k * n * R > (1LL << 28) || m * n * R > (1LL << 28))
    return fail(FM_E_UNSUPPORTED, "Kronecker power too large");
  *out = clone(power(*s, levels));
  return *out ? FM_OK : fail(FM_E_NOMEM, "out of host memory");
} catch (...) {
  return host_failure();
}

int fm_scheme_dims(const fm_scheme* s, int* m, int* n, int* k, int* R) try {
  clear_error();
  if (!s) return fail(FM_E_ARG, "null scheme");
  if (m) *m = s->m;
  if (n) *n = s->n;
  if (k) *k = s->k;
  if (R) *R = s->R;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_scheme_coeffs(const fm_scheme* s, double* U, double* V, double* W) try {
  clear_error();
  if (!s || !U || !V || !W) return fail(FM_E_ARG, "null pointer");
  std::copy(s->U.begin(), s->U.end(), U);
  std::copy(s->V.begin(), s->V.end(), V);
  std::copy(s->W.begin(), s->W.end(), W);
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_scheme_coeffs_f32(const fm_scheme* s, int levels, float* U, float* V, float* W) try {
  clear_error();
  if (!s || !U || !V || !W) return fail(FM_E_ARG, "null pointer");
  if (levels < 1 || levels > 8) return fail(FM_E_ARG, "levels must be in [1, 8]");
  const fm_scheme f = power(*s, levels);
  for (size_t i = 0; i < f.U.size(); ++i) U[i] = (float)f.U[i];
  for (size_t i = 0; i < f.V.size(); ++i) V[i] = (float)f.V[i];
  for (size_t i = 0; i < f.W.size(); ++i) W[i] = (float)f.W[i];
  return FM_OK;
} catch (...) {
  return host_failure();
}

void fm_scheme_free(fm_scheme* s) { delete s; }

static int scale_mode_ok(int m) {
  const int b = m & 0xff, flags = m & ~0xff;
  if (b != FM_SCALE_TENSOR && b != FM_SCALE_ROWCOL && b != FM_SCALE_GROUP) return 0;
  if (flags & ~(FM_REPAIR_ROWS | FM_REPAIR_WEIGHTS)) return 0;
  return !flags || b == FM_SCALE_GROUP;  // the repairs belong to the group schedule
}

size_t fm_workspace_size_scaled(const fm_scheme* s, int M, int N, int K, int levels, int G,
                                int chunk, fm_scale_mode scale_mode) try {
  Geometry g;
  if (G < 1 || !scale_mode_ok(scale_mode) || check_geometry(s, levels, M, N, K, g) != FM_OK ||
      scale_shape_ok(g.Mb, g.Nb, g.Kb, g.R, scale_mode) != FM_OK)
    return 0;
  if (chunk <= 0 || chunk > G) chunk = G;
  return make_layout(g, G, chunk, true, scale_mode, chunk < G).total;
} catch (...) {
  return host_failure(), (size_t)0;
}

size_t fm_workspace_size(const fm_scheme* s, int M, int N, int K, int levels, int G, int chunk) try {
  return fm_workspace_size_scaled(s, M, N, K, levels, G, chunk, FM_SCALE_TENSOR);
} catch (...) {
  return host_failure(), (size_t)0;
}

size_t fm_error_workspace_size(int M, int N) try {
  if (M < 1 || N < 1) return 0;
  const size_t n = (size_t)M * N;
  return up((size_t)error_stats_blocks(n) * 3 * 8) + up(3 * 8);
} catch (...) {
  return host_failure(), (size_t)0;
}

int fm_form_operands_scaled(const fm_scheme* s, int levels, const float* A, const float* B,
                            int M, int N, int K, fm_fmt fmt, fm_scale_mode scale_mode, uint8_t* Tq,
                            uint8_t* Sq, float* dT, float* dS, void* workspace, size_t ws_bytes,
                            void* hip_stream) try {
  clear_error();
  if (!A || !B || !Tq || !Sq || !dT || !dS) return fail(FM_E_ARG, "null pointer");
  if (!fmt_ok(fmt)) return fail(FM_E_ARG, "bad format");
  if (!scale_mode_ok(scale_mode)) return fail(FM_E_ARG, "bad scale mode");
  Geometry geo;
  if (int rc = check_geometry(s, levels, M, N, K, geo)) return rc;
  if (int rc = scale_shape_ok(geo.Mb, geo.Nb, geo.Kb, geo.R, scale_mode)) return rc;
  const Layout L = make_layout(geo, 1, 1, true, scale_mode);
  if (int rc = check_ws(workspace, ws_bytes, L.total)) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  char* ws = (char*)workspace;
  int rc = FM_OK;
  const fm_scheme* one[1] = {s};
  Tables T = make_tables(one, 1, levels, geo, rc);
  if (rc) return rc;
  if ((rc = upload_tables(T, ws, L, st))) return rc;
  float* Bt = (float*)(ws + L.bt);
  if ((rc = launch_transpose(B, Bt, K, N, st))) return rc;
  const float *Aform, *rowup;
  if ((rc = prepare_repairs(geo, T, ws, L, scale_mode, A, Aform, rowup, st))) return rc;
  return form_chunk(geo, Aform, Bt, ws, L, T, 0, 1, fmt, scale_mode, Tq, Sq, dT, dS, st);
} catch (...) {
  return host_failure();
}

int fm_form_operands(const fm_scheme* s, int levels, const float* A, const float* B, int M, int N,
                     int K, fm_fmt fmt, uint8_t* Tq, uint8_t* Sq, float* dT, float* dS,
                     void* workspace, size_t ws_bytes, void* hip_stream) try {
  return fm_form_operands_scaled(s, levels, A, B, M, N, K, fmt, FM_SCALE_TENSOR, Tq, Sq, dT, dS,
                                 workspace, ws_bytes, hip_stream);
} catch (...) {
  return host_failure();
}

int fm_block_products_scaled(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                             const float* dS, int batch, int Mb, int Nb, int Kb, fm_fmt fmt,
                             fm_scale_mode scale_mode, float* Mout, void* hip_stream) try {
  clear_error();
  if (!Tq || !Sq || !dT || !dS || !Mout) return fail(FM_E_ARG, "null pointer");
  if (!fmt_ok(fmt)) return fail(FM_E_ARG, "bad format");
  if (!scale_mode_ok(scale_mode) || (scale_mode & ~0xff))
    return fail(FM_E_ARG, "bad scale mode (the repairs act on the operands, not on the products)");
  if (batch < 1 || Mb < 1 || Nb < 1 || Kb < 1) return fail(FM_E_ARG, "sizes must be positive");
  if (Kb % 16) return fail(FM_E_SHAPE, "Kb must be a multiple of 16");
  // scales read in aligned 16-byte chunks (float4 column scales; group
  // scales as the chunk holding the entry)
  auto aligned16 = [](const void* p) { return ((uintptr_t)p & 15u) == 0; };
  if (scale_mode == FM_SCALE_ROWCOL && !aligned16(dS))
    return fail(FM_E_ARG, "per-column scales must be 16-byte aligned");
  if (scale_mode == FM_SCALE_GROUP && (!aligned16(dT) || !aligned16(dS)))
    return fail(FM_E_ARG, "group scales must be 16-byte aligned (and padded to 4 floats)");
  return launch_block_gemm(Tq, Sq, dT, dS, Mout, batch, Mb, Nb, Kb, fmt, scale_mode,
                           (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

int fm_block_products(const uint8_t* Tq, const uint8_t* Sq, const float* dT, const float* dS,
                      int batch, int Mb, int Nb, int Kb, fm_fmt fmt, float* Mout,
                      void* hip_stream) try {
  return fm_block_products_scaled(Tq, Sq, dT, dS, batch, Mb, Nb, Kb, fmt, FM_SCALE_TENSOR, Mout,
                                  hip_stream);
} catch (...) {
  return host_failure();
}

int fm_reconstruct(const fm_scheme* s, int levels, const float* Mprod, int M, int N, float* C,
                   void* workspace, size_t ws_bytes, void* hip_stream) try {
  clear_error();
  if (!Mprod || !C) return fail(FM_E_ARG, "null pointer");
  Geometry geo;
  // K does not matter for the reconstruction; use the grid's k^L (Kb = 16).
  long long gk = 1;
  if (s)
    for (int l = 0; l < levels && gk <= 64; ++l) gk *= s->k;
  if (int rc = check_geometry(s, levels, M, N, (int)std::min<long long>(gk, 64) * 16, geo)) return rc;
  const Layout L = make_layout(geo, 1, 1, false);
  if (int rc = check_ws(workspace, ws_bytes, L.total)) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  char* ws = (char*)workspace;
  int rc = FM_OK;
  const fm_scheme* one[1] = {s};
  Tables T = make_tables(one, 1, levels, geo, rc);
  if (rc) return rc;
  if ((rc = upload_tables(T, ws, L, st))) return rc;
  const ReconArgs ra = recon_args(geo, ws, L, 0, 1, Mprod, C, nullptr);
  return launch_recon(ra, chunk_pattern(T, 2, 0, 1), st);
} catch (...) {
  return host_failure();
}

int fm_matmul_lowp_scaled(const fm_scheme* s, const float* A, const float* B, float* C, int M,
                          int N, int K, int levels, fm_fmt fmt, fm_scale_mode scale_mode,
                          void* workspace, size_t ws_bytes, void* hip_stream) try {
  clear_error();
  if (!A || !B || !C) return fail(FM_E_ARG, "null pointer");
  if (!fmt_ok(fmt)) return fail(FM_E_ARG, "bad format");
  if (!scale_mode_ok(scale_mode)) return fail(FM_E_ARG, "bad scale mode");
  Geometry geo;
  if (int rc = check_geometry(s, levels, M, N, K, geo)) return rc;
  if (int rc = scale_shape_ok(geo.Mb, geo.Nb, geo.Kb, geo.R, scale_mode)) return rc;
  const Layout L = make_layout(geo, 1, 1, true, scale_mode);
  if (int rc = check_ws(workspace, ws_bytes, L.total)) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  char* ws = (char*)workspace;
  int rc = FM_OK;
  const fm_scheme* one[1] = {s};
  Tables T = make_tables(one, 1, levels, geo, rc);
  if (rc) return rc;
  if ((rc = upload_tables(T, ws, L, st))) return rc;
  float* Bt = (float*)(ws + L.bt);
  if ((rc = launch_transpose(B, Bt, K, N, st))) return rc;
  uint8_t* Tq = (uint8_t*)(ws + L.tq);
  uint8_t* Sq = (uint8_t*)(ws + L.sq);
  const float *Aform, *rowup;
  if ((rc = prepare_repairs(geo, T, ws, L, scale_mode, A, Aform, rowup, st))) return rc;
  if ((rc = form_chunk(geo, Aform, Bt, ws, L, T, 0, 1, fmt, scale_mode, Tq, Sq, nullptr, nullptr,
                       st)))
    return rc;
  const float* dd = (const float*)(ws + L.d);
  float* Mp = (float*)(ws + L.mprod);
  timing_begin(T_BLOCK_GEMM, st);
  // group scales return bf16 products: stored as bf16 on the way to the
  // reconstruction (half the bytes, the same values)
  const bool bf = base_mode(scale_mode) == FM_SCALE_GROUP;
  if ((rc = launch_block_gemm(Tq, Sq, dd, dd + (size_t)geo.R * scales_a(geo, scale_mode), Mp,
                              geo.R, geo.Mb, geo.Nb, geo.Kb, fmt, base_mode(scale_mode), st, bf)))
    return rc;
  timing_end(T_BLOCK_GEMM, st);
  ReconArgs ra = recon_args(geo, ws, L, 0, 1, Mp, C, nullptr);
  ra.rowscale = rowup;
  ra.prod_bf16 = bf;
  return launch_recon(ra, chunk_pattern(T, 2, 0, 1), st);
} catch (...) {
  return host_failure();
}

int fm_matmul_lowp(const fm_scheme* s, const float* A, const float* B, float* C, int M, int N,
                   int K, int levels, fm_fmt fmt, void* workspace, size_t ws_bytes,
                   void* hip_stream) try {
  return fm_matmul_lowp_scaled(s, A, B, C, M, N, K, levels, fmt, FM_SCALE_TENSOR, workspace,
                               ws_bytes, hip_stream);
} catch (...) {
  return host_failure();
}

int fm_reference_f64(const float* A, const float* B, double* C_ref, int M, int N, int K,
                     void* hip_stream) try {
  clear_error();
  if (!A || !B || !C_ref) return fail(FM_E_ARG, "null pointer");
  if (M < 1 || N < 1 || K < 1) return fail(FM_E_ARG, "sizes must be positive");
  timing_begin(T_REFERENCE, (hipStream_t)hip_stream);
  const int rc = launch_reference_f64(A, B, C_ref, M, N, K, (hipStream_t)hip_stream);
  timing_end(T_REFERENCE, (hipStream_t)hip_stream);
  return rc;
} catch (...) {
  return host_failure();
}

int fm_error_stats(const float* C, const double* C_ref, int M, int N, fm_stats* out,
                   void* workspace, size_t ws_bytes, void* hip_stream) try {
  clear_error();
  if (!C || !C_ref || !out) return fail(FM_E_ARG, "null pointer");
  if (M < 1 || N < 1) return fail(FM_E_ARG, "sizes must be positive");
  const size_t n = (size_t)M * N;
  if (int rc = check_ws(workspace, ws_bytes, fm_error_workspace_size(M, N))) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  char* ws = (char*)workspace;
  const int nblk = error_stats_blocks(n);
  double* partial = (double*)ws;
  double* out3 = (double*)(ws + up((size_t)nblk * 3 * 8));
  if (int rc = launch_error_stats(C, C_ref, n, partial, st)) return rc;
  if (int rc = launch_error_finalize(partial, nblk, out3, st)) return rc;
  double h[3];
  if (int rc = download(h, out3, sizeof(h), st)) return rc;
  out->err_sq = h[0];
  out->ref_sq = h[1];
  out->max_abs = h[2];
  out->rel_fro = h[1] > 0 ? std::sqrt(h[0]) / std::sqrt(h[1]) : 0.0;
  if (!std::isfinite(h[0])) return fail(FM_E_NONFINITE, "non-finite error sum");
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_orbit_eval_scaled(const fm_scheme* const* gauged, int G, const float* A, const float* B,
                         const double* C_ref, int M, int N, int K, int levels, fm_fmt fmt,
                         fm_scale_mode scale_mode, double* rel_fro_out, void* workspace,
                         size_t ws_bytes, void* hip_stream) try {
  clear_error();
  if (!gauged || !A || !B || !C_ref || !rel_fro_out) return fail(FM_E_ARG, "null pointer");
  if (G < 1) return fail(FM_E_ARG, "G must be positive");
  if (!fmt_ok(fmt)) return fail(FM_E_ARG, "bad format");
  if (!scale_mode_ok(scale_mode)) return fail(FM_E_ARG, "bad scale mode");
  Geometry geo;
  if (int rc = check_geometry(gauged[0], levels, M, N, K, geo)) return rc;
  if (int rc = scale_shape_ok(geo.Mb, geo.Nb, geo.Kb, geo.R, scale_mode)) return rc;
  // the largest chunk of gauges that fits, halving from G; with several
  // chunks, two sets of maxima, scales and block products if they fit (the
  // reconstruction of one chunk then runs beside the next chunk's formation,
  // and per-tensor maxima are formed a chunk ahead)
  int chunk = G;
  Layout L = make_layout(geo, G, chunk, true, scale_mode);
  while (chunk > 1 && L.total > ws_bytes) {
    chunk = std::max(1, chunk / 2);
    L = make_layout(geo, G, chunk, true, scale_mode, true);
    if (L.total > ws_bytes) L = make_layout(geo, G, chunk, true, scale_mode);
  }
  if (int rc = check_ws(workspace, ws_bytes, L.total)) return rc;
  hipStream_t st = (hipStream_t)hip_stream;
  Pipeline pipe;
  static const bool one_stream = [] {
    const char* e = std::getenv("FM_ORBIT_STREAMS");
    return e && std::strcmp(e, "1") == 0;
  }();
  if (L.two_sets() && !one_stream) {
    if (int rc = pipe.open(st)) return rc;
  }
  char* ws = (char*)workspace;
  int rc = FM_OK;
  // Coefficient tables: with several chunks (and no joint rounding, whose
  // set-up needs every gauge's tables), those of the first two chunks are
  // built and uploaded first, the rest while the first chunk runs on the
  // device.  Every gauge's grid and rank are checked before any device work.
  for (int g = 0; g < G; ++g) {
    const fm_scheme* s = gauged[g];
    if (!s) return fail(FM_E_ARG, "null scheme in orbit");
    long long m = 1, k = 1, n = 1, R = 1;
    for (int l = 0; l < levels; ++l) {
      m *= s->m;
      k *= s->k;
      n *= s->n;
      R *= s->R;
    }
    if (m != geo.gm || k != geo.gk || n != geo.gn || R != geo.R)
      return fail(FM_E_MISMATCH, "schemes of one orbit must share grid and rank");
  }
  const int G1 = (L.two_sets() && !repair_weights(scale_mode)) ? std::min(G, 2 * chunk) : G;
  Tables T;
  if ((rc = extend_tables(T, gauged, 0, G1, levels, geo))) return rc;
  if (G1 < G) {
    // staging for the largest upload (dense lists) up front: no pinned
    // allocation while the orbit runs
    const size_t per_gauge = (size_t)(geo.R + 1) * 4 * 3 +
                             (size_t)geo.R * (geo.NBa() + geo.NBb() + geo.NC()) * 8;
    if ((rc = stage_reserve(per_gauge * (size_t)G))) return rc;
    if ((rc = upload_table_range(T, ws, L, 0, G1, st))) return rc;
  } else if ((rc = upload_tables(T, ws, L, st))) {
    return rc;
  }
  if ((rc = launch_fill_u32((uint32_t*)(ws + L.flags), 1, 0u, st))) return rc;
  float* Bt = (float*)(ws + L.bt);
  if ((rc = launch_transpose(B, Bt, K, N, st))) return rc;
  uint8_t* Tq = (uint8_t*)(ws + L.tq);
  uint8_t* Sq = (uint8_t*)(ws + L.sq);
  float* Mp = (float*)(ws + L.mprod);
  double* errsq = (double*)(ws + L.errsq);
  const float *Aform, *rowup;
  if ((rc = prepare_repairs(geo, T, ws, L, scale_mode, A, Aform, rowup, st))) return rc;
  // group scales return bf16 products: stored as bf16 on the way to the
  // reconstruction (half the bytes, the same values)
  const bool bf = base_mode(scale_mode) == FM_SCALE_GROUP;
  // per-tensor scales over several chunks: each chunk's codes are formed
  // together with the next chunk's maxima (chunk 0's maxima first)
  const bool fuse = L.two_sets() && scale_mode == FM_SCALE_TENSOR;
  if (fuse) {
    const int n0 = std::min(chunk, G);
    FormArgs fa, fb;
    tensor_form_args(geo, Aform, Bt, ws, L, 0, n0, fmt, Tq, Sq, fa, fb);
    set_trie(fa, T, ws, L, 0, 0, n0);
    set_trie(fb, T, ws, L, 1, 0, n0);
    if ((rc = launch_fill_u32(fa.amax, (size_t)2 * n0 * geo.R, 0u, st))) return rc;
    for (int side = 0; side < 2; ++side) {
      timing_begin(T_FORM_AMAX, st);
      if ((rc = launch_form(side ? fb : fa, 0, chunk_pattern(T, side, 0, n0), side, st))) return rc;
      timing_end(T_FORM_AMAX, st);
    }
    if ((rc = launch_scales(fa.amax, (float*)(ws + L.q), (float*)(ws + L.d), 2 * n0 * geo.R, fmt,
                            (uint32_t*)(ws + L.flags), st)))
      return rc;
  }
  for (int g0 = 0, c = 0; g0 < G; g0 += chunk, ++c) {
    const int n = std::min(chunk, G - g0);
    // chunk c uses set c mod 2 (maxima, scales, products) when there are two
    const int buf = L.two_sets() ? (c & 1) : 0;
    const Layout Lc = L.set(buf);
    float* Mc = (float*)(ws + Lc.mprod);
    const float* dd = (const float*)(ws + Lc.d);
    if (fuse) {
      const int n1 = std::min(chunk, std::max(0, G - g0 - n));
      if ((rc = form_codes_and_next_maxima(geo, Aform, Bt, ws, L, T, c, g0, n, n1, fmt, Tq, Sq,
                                           st)))
        return rc;
    } else if ((rc = form_chunk(geo, Aform, Bt, ws, Lc, T, g0, n, fmt, scale_mode, Tq, Sq,
                                nullptr, nullptr, st))) {
      return rc;
    }
    // the previous chunk's reconstruction runs beside this chunk's
    // formation and is done before these products start: the block
    // products, the bulk of the work, then have the GPU to themselves (a
    // reconstruction running beside them slows them more than it gains)
    if (c >= 1 && (rc = pipe.wait_reconstructed(buf ^ 1))) return rc;
    // products of whole tiles go to the reconstruction in the tiled layout
    // (contiguous stores) when a family kernel reconstructs them
    const int rpat = chunk_pattern(T, 2, g0, n);
    const int trows = block_gemm_tile_rows(geo.Mb, geo.Nb, geo.Kb, base_mode(scale_mode), bf);
    const bool tiled = scale_mode == FM_SCALE_TENSOR && rpat >= 0 && trows > 0 &&
                       geo.Mb % trows == 0 && geo.Nb % 128 == 0 && geo.N % 4 == 0 &&
                       geo.gm * geo.gn <= 64 && (size_t)geo.R * geo.Mb * geo.Nb * 4 < ((size_t)1 << 32);
    timing_begin(T_BLOCK_GEMM, st);
    if ((rc = launch_block_gemm(Tq, Sq, dd, dd + (size_t)n * geo.R * scales_a(geo, scale_mode), Mc,
                                n * geo.R, geo.Mb, geo.Nb, geo.Kb, fmt, base_mode(scale_mode),
                                st, bf, tiled)))
      return rc;
    timing_end(T_BLOCK_GEMM, st);
    hipStream_t rs = st;
    if (pipe.on && (rc = pipe.hand_over(buf, rs))) return rc;
    ReconArgs ra = recon_args(geo, ws, Lc, g0, n, Mc, nullptr, C_ref);
    ra.rowscale = rowup;
    ra.prod_bf16 = bf;
    ra.tiled = tiled ? trows : 0;
    const int nblk = recon_blocks(ra);
    timing_begin(T_RECON, rs);
    if ((rc = launch_recon(ra, rpat, rs))) return rc;
    timing_end(T_RECON, rs);
    if ((rc = launch_reduce_rows((double*)(ws + L.partial), nblk, n, errsq + g0, rs))) return rc;
    if (pipe.on && (rc = pipe.reconstructed(buf))) return rc;
    // the remaining gauges' tables, built while the first chunk runs; they
    // are uploaded on the caller's stream ahead of the next formation pass,
    // the first to read them (chunk 2's maxima)
    if (c == 0 && T.G < G) {
      const int Gd = T.G;
      if ((rc = extend_tables(T, gauged, Gd, G, levels, geo))) return rc;
      if ((rc = upload_table_range(T, ws, L, Gd, G, st))) return rc;
    }
  }
  if ((rc = pipe.join())) return rc;
  // sum of squares of the reference (err_sq of a zero output)
  {
    const size_t nel = (size_t)M * N;
    const int nblk = error_stats_blocks(nel);
    // reuse the product buffer as scratch for the partial sums
    double* partial = (double*)Mp;
    if ((size_t)nblk * 3 * 8 > (size_t)chunk * geo.R * geo.Mb * geo.Nb * 4)
      return fail(FM_E_WORKSPACE, "workspace too small for the reference norm");
    if ((rc = launch_error_stats(nullptr, C_ref, nel, partial, st))) return rc;
    if ((rc = launch_error_finalize(partial, nblk, (double*)(ws + L.out3), st))) return rc;
  }
  std::vector<double> h((size_t)G + 3 + 1);
  if ((rc = download(h.data(), errsq, (size_t)G * 8, st))) return rc;
  double o3[3];
  if ((rc = download(o3, ws + L.out3, sizeof(o3), st))) return rc;
  uint32_t flag = 0;
  if ((rc = download(&flag, ws + L.flags, 4, st))) return rc;
  if (flag) return fail(FM_E_NONFINITE, "a block sum was not finite");
  const double ref = std::sqrt(o3[1]);
  for (int g = 0; g < G; ++g) rel_fro_out[g] = ref > 0 ? std::sqrt(h[g]) / ref : 0.0;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_orbit_eval(const fm_scheme* const* gauged, int G, const float* A, const float* B,
                  const double* C_ref, int M, int N, int K, int levels, fm_fmt fmt,
                  double* rel_fro_out, void* workspace, size_t ws_bytes, void* hip_stream) try {
  return fm_orbit_eval_scaled(gauged, G, A, B, C_ref, M, N, K, levels, fmt, FM_SCALE_TENSOR,
                              rel_fro_out, workspace, ws_bytes, hip_stream);
} catch (...) {
  return host_failure();
}

int fm_set_block_product_arithmetic(fm_accum a) try {
  clear_error();
  return set_block_product_arith((int)a);
} catch (...) {
  return host_failure();
}

int fm_fp8_encode(const float* x, int64_t n, fm_fmt fmt, int impl, uint8_t* out,
                  void* hip_stream) try {
  clear_error();
  if (!x || !out) return fail(FM_E_ARG, "null pointer");
  if (n < 0 || impl < 0 || impl > 2 || !fmt_ok(fmt)) return fail(FM_E_ARG, "bad argument");
  return launch_fp8_encode(x, out, (size_t)n, fmt, impl, (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

int fm_bf16_round(const float* x, int64_t n, int impl, float* out, void* hip_stream) try {
  clear_error();
  if (!x || !out) return fail(FM_E_ARG, "null pointer");
  if (n < 0 || impl < 0 || impl > 2) return fail(FM_E_ARG, "bad argument");
  if ((uint64_t)n > ((uint64_t)0xffffffffu) * 256u) return fail(FM_E_SHAPE, "too many values");
  return launch_bf16_round(x, out, (size_t)n, impl, (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

const char* fm_scheme_kernel_family(const fm_scheme* s, int levels) try {
  clear_error();
  if (!s || levels < 1 || levels > 8) {
    fail(FM_E_ARG, "bad argument");
    return "";
  }
  const fm_scheme f = power(*s, levels);
  Lists L;
  build_lists(f, L);
  const int pa = match_pattern(0, L.a, f.R, f.m * f.k);
  const int pb = match_pattern(1, L.b, f.R, f.n * f.k);
  const int pw = match_pattern(2, L.w, f.R, f.m * f.n);
  if (pa >= 0 && pa == pb && pb == pw) return pattern_name(pa);
  return "generic";
} catch (...) {
  return host_failure(), "";
}

int fm_scheme_sign_variant(const fm_scheme* s, int levels, int side, int* is_sign,
                           uint64_t* neg_mask) try {
  clear_error();
  if (!s || !is_sign || !neg_mask) return fail(FM_E_ARG, "null pointer");
  if (side < 0 || side > 1) return fail(FM_E_ARG, "side must be 0 (A) or 1 (B)");
  if (levels < 1 || levels > 8) return fail(FM_E_ARG, "levels must be in [1, 8]");
  const fm_scheme f = power(*s, levels);
  Lists L;
  build_lists(f, L);
  const Side& sd = side ? L.b : L.a;
  const int nb = side ? f.n * f.k : f.m * f.k;
  const int p = match_pattern(side, sd, f.R, nb);
  uint64_t m = 0;
  *is_sign = block_signs(p, side, sd, nb, &m) ? 1 : 0;
  *neg_mask = *is_sign ? m : 0;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_timing_enable(int on) try {
  clear_error();
  g_timing.on = on != 0;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_timing_reset(void) try {
  clear_error();
  for (auto& r : g_timing.recs) {
    (void)hipEventSynchronize(r.stop);
    g_timing.pool.push_back(r.start);
    g_timing.pool.push_back(r.stop);
  }
  g_timing.recs.clear();
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_timing_read(const char* kernel_class, int* launches, double* total_ms) try {
  clear_error();
  if (!kernel_class || !launches || !total_ms) return fail(FM_E_ARG, "null pointer");
  int cls = -1;
  for (int c = 0; c < T_COUNT; ++c)
    if (std::strcmp(kernel_class, kTimedNames[c]) == 0) cls = c;
  if (cls < 0) return fail(FM_E_ARG, std::string("unknown kernel class ") + kernel_class);
  int n = 0;
  double ms = 0.0;
  for (auto& r : g_timing.recs) {
    if (r.cls != cls) continue;
    if (int rc = hip_check(hipEventSynchronize(r.stop), "hipEventSynchronize")) return rc;
    float t = 0.f;
    if (int rc = hip_check(hipEventElapsedTime(&t, r.start, r.stop), "hipEventElapsedTime"))
      return rc;
    ms += t;
    ++n;
  }
  *launches = n;
  *total_ms = ms;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_status(void* workspace, size_t ws_bytes, void* hip_stream) try {
  clear_error();
  if (!workspace || ws_bytes < kAlign) return fail(FM_E_WORKSPACE, "workspace too small");
  hipStream_t st = (hipStream_t)hip_stream;
  uint32_t flag = 0;
  if (int rc = download(&flag, workspace, 4, st)) return rc;
  if (int rc = launch_fill_u32((uint32_t*)workspace, 1, 0u, st)) return rc;
  if (flag & 2u) return fail(FM_E_RANGE, "a block sum of integer codes left int8");
  if (flag) return fail(FM_E_NONFINITE, "a block sum was not finite");
  return FM_OK;
} catch (...) {
  return host_failure();
}

// ------------------------------------------------------------ integer path
int fm_int8_quantize(const float* X, int rows, int K, int g, int b, int8_t* codes, float* d,
                     uint32_t* flag, void* hip_stream) try {
  clear_error();
  if (!X || !codes || !d) return fail(FM_E_ARG, "null pointer");
  if (rows < 1 || K < 1) return fail(FM_E_ARG, "sizes must be positive");
  if (b < 1 || b > 127) return fail(FM_E_ARG, "code bound must be in [1, 127]");
  if (g < 64 || g > 512 || g % 64) return fail(FM_E_ARG, "group length must be 64..512, a multiple of 64");
  if (K % g) return fail(FM_E_SHAPE, "K must be a multiple of the group length");
  return launch_i8_quantize(X, rows, K, g, b, codes, d, flag, (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

int fm_int8_matmul_classical(const int8_t* Ac, const float* dA, const int8_t* BTc, const float* dB,
                             int M, int N, int K, int g, float* out, void* hip_stream) try {
  clear_error();
  if (!Ac || !dA || !BTc || !dB || !out) return fail(FM_E_ARG, "null pointer");
  if (M < 1 || N < 1 || K < 1) return fail(FM_E_ARG, "sizes must be positive");
  if (g < 128 || g % 128 || K % g) return fail(FM_E_SHAPE, "g must be a multiple of 128 dividing K");
  if (M % 4 || N % 4) return fail(FM_E_SHAPE, "M and N must be multiples of 4");
  return launch_i8_gemm(false, Ac, BTc, nullptr, nullptr, dA, dB, out, nullptr, nullptr, 0,
                        nullptr, nullptr, 0, M, N, K, g, 1, 1, 1, 0, 1, nullptr, nullptr, nullptr,
                        nullptr, (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

namespace {
// The flattened scheme's integer tables and certificate quantities.
struct IntScheme {
  int gm = 0, gk = 0, gn = 0, R = 0;
  std::vector<int> U, V, W;
  double LA = 0, LB = 0, LW = 0;
};

int int_scheme(const fm_scheme* s, int levels, IntScheme& out) {
  if (!s) return fail(FM_E_ARG, "null scheme");
  if (levels < 1 || levels > 3) return fail(FM_E_ARG, "levels must be 1..3");
  const fm_scheme f = levels > 1 ? power(*s, levels) : *s;
  out.gm = f.m;
  out.gk = f.k;
  out.gn = f.n;
  out.R = f.R;
  auto conv = [&](const std::vector<double>& x, std::vector<int>& y) {
    y.resize(x.size());
    for (size_t i = 0; i < x.size(); ++i) {
      if (x[i] != std::floor(x[i]) || std::fabs(x[i]) > 127) return false;
      y[i] = (int)x[i];
    }
    return true;
  };
  if (!conv(f.U, out.U) || !conv(f.V, out.V) || !conv(f.W, out.W))
    return fail(FM_E_ARG, "coefficients are not small integers");
  const int R = f.R, na = f.m * f.k, nb = f.k * f.n, nc = f.m * f.n;
  out.LA = out.LB = out.LW = 0;
  for (int r = 0; r < R; ++r) {
    double a = 0, b = 0;
    for (int i = 0; i < na; ++i) a += std::abs(out.U[(size_t)r * na + i]);
    for (int i = 0; i < nb; ++i) b += std::abs(out.V[(size_t)r * nb + i]);
    out.LA = std::max(out.LA, a);
    out.LB = std::max(out.LB, b);
  }
  for (int c = 0; c < nc; ++c) {
    double w = 0;
    for (int r = 0; r < R; ++r) w += std::abs(out.W[(size_t)r * nc + c]);
    out.LW = std::max(out.LW, w);
  }
  return FM_OK;
}

void certify(const IntScheme& is, int bA, int bB, int h, int g, int cond[3]) {
  const double alpha = is.LA * bA, beta = is.LB * bB;
  cond[0] = alpha <= 127 && beta <= 127;
  cond[1] = std::max(is.LW * h * alpha * beta, (double)g * bA * bB) < 2147483648.0;
  cond[2] = h > 0 && g % (is.gk * h) == 0;
}

// The corrected computation's certificate (App. D, generalized from two-level
// Strassen at code bound 127): block sums reach at most alpha = L_A b_A, so
// the split parts satisfy |q| <= qmax = floor((alpha + 128) / 256) and
// remainders lie in [-128, 127]; every weighted scalar term of eq. (2) for an
// output entry adds up to at most L_W h (128 + 256 qmax_A)(128 + 256 qmax_B),
// which must stay below 2^31 (condition 1; it bounds every partial sum in
// any order), with the split parts within int8 (condition 0) and a call
// inside one group (condition 2).  bound[0] is that sum, bound[1..2] qmax.
int corr_qmax(double alpha) { return (int)std::floor((alpha + 128.0) / 256.0); }
void certify_corrected(const IntScheme& is, int bA, int bB, int h, int g, int cond[3],
                       double bound[3]) {
  const int qa = corr_qmax(is.LA * bA), qb = corr_qmax(is.LB * bB);
  bound[0] = is.LW * h * (128.0 + 256.0 * qa) * (128.0 + 256.0 * qb);
  bound[1] = qa;
  bound[2] = qb;
  cond[0] = qa <= 127 && qb <= 127;
  cond[1] = std::max(bound[0], (double)g * bA * bB) < 2147483648.0;
  cond[2] = h > 0 && g % (is.gk * h) == 0;
}

// Bytes per product in a block-sum coefficient table: the blocks' int8
// coefficients, zero-padded to whole dwords.
int coef_stride(int blocks) { return (blocks + 3) / 4 * 4; }

// Fast-path workspace: flags, a zero segment, coefficient tables, segment
// tables, the tile schedule, then per call the block sums T (R x Mb x h), S
// and -S (R x Nb x h).
struct I8Layout {
  size_t flags, zero, coefa, coefb, segs, segoff, order, order_off, phase, t, s, sn, tr, sr, snr,
      total;
  int nsegs;
};

// Segments of one output block per call: its n nonzero weights once
// (padded to whole K steps), or with the correction in three phases of n,
// 2 n and n segments, each padded.
int block_segments(int n, int per_step, bool corr) {
  auto pad = [&](int k) { return (k + per_step - 1) / per_step * per_step; };
  return corr ? 2 * pad(n) + pad(2 * n) : pad(n);
}

I8Layout i8_layout(const IntScheme& is, int M, int N, int K, int h, bool corr) {
  I8Layout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += up(bytes);
    return at;
  };
  const int per_step = 128 / h;
  int nsegs = 0;
  for (int c = 0; c < is.gm * is.gn; ++c) {
    int n = 0;
    for (int r = 0; r < is.R; ++r) n += is.W[(size_t)r * is.gm * is.gn + c] != 0;
    nsegs += block_segments(n, per_step, corr);
  }
  L.nsegs = nsegs;
  const size_t ncall = (size_t)K / ((size_t)is.gk * h);
  L.flags = take(kAlign);
  L.zero = take(kAlign);
  L.coefa = take((size_t)is.R * coef_stride(is.gm * is.gk));
  L.coefb = take((size_t)is.R * coef_stride(is.gn * is.gk));
  L.segs = take((size_t)nsegs * 4);
  L.segoff = take((size_t)(is.gm * is.gn + 1) * 4);
  L.order = take((size_t)i8_fast_tiles(is.gm, is.gn, M / is.gm, N / is.gn) * 4);
  L.order_off = take(257 * 4);
  L.phase = take((size_t)is.gm * is.gn * 2 * 4);
  const size_t tb = ncall * is.R * (M / is.gm) * h, sb = ncall * is.R * (N / is.gn) * h;
  L.t = take(tb);
  L.s = take(sb);
  L.sn = take(sb);
  L.tr = corr ? take(tb) : 0;
  L.sr = corr ? take(sb) : 0;
  L.snr = corr ? take(sb) : 0;
  L.total = o;
  return L;
}

int i8_fast_shape_ok(const IntScheme& is, int M, int N, int K, int g, int h) {
  if (M < 1 || N < 1 || K < 1) return fail(FM_E_ARG, "sizes must be positive");
  if (h < 16 || h > 128 || h % 16 || 128 % h) return fail(FM_E_ARG, "h must be 16, 32, 64 or 128");
  if (g < 128 || g % 128 || K % g) return fail(FM_E_SHAPE, "g must be a multiple of 128 dividing K");
  if (M % (4 * is.gm) || N % (4 * is.gn))
    return fail(FM_E_SHAPE, "M and N must be multiples of 4 m^L and 4 n^L");
  if (is.gm * is.gn > 64) return fail(FM_E_UNSUPPORTED, "output grid larger than 64 blocks");
  return FM_OK;
}

// Validation, certificate, tables and schedule of a fast call (everything
// that depends on the scheme and the shapes, not on the codes): the tables
// go to the workspace with one staged copy on st.  corr selects the overflow
// correction (eq. (2)).
int i8_plan_prepare(const fm_scheme* s, int levels, int M, int N, int K, int g, int h, int b_A,
                    int b_B, bool corr, void* workspace, size_t ws_bytes, hipStream_t st,
                    fm_int8_plan& p) {
  IntScheme is;
  if (int rc = int_scheme(s, levels, is)) return rc;
  if (int rc = i8_fast_shape_ok(is, M, N, K, g, h)) return rc;
  if (b_A < 1 || b_A > 127 || b_B < 1 || b_B > 127) return fail(FM_E_ARG, "code bounds must be in [1, 127]");
  const int calls_per_group = g / (is.gk * h);
  int qa = 0, qb = 0;
  if (corr) {
    int cond[3];
    double bound[3];
    certify_corrected(is, b_A, b_B, h, g, cond, bound);
    if (!cond[0]) return fail(FM_E_UNCERTIFIED, "the split parts of a block sum leave int8");
    if (!cond[1]) return fail(FM_E_UNCERTIFIED, "a corrected partial sum can leave int32");
    if (!cond[2]) return fail(FM_E_UNCERTIFIED, "condition (iii): a call spans two groups");
    if (calls_per_group != 1)
      return fail(FM_E_UNSUPPORTED, "the corrected kernel needs one call per group (g = k^levels h)");
    qa = (int)bound[1];
    qb = (int)bound[2];
  } else {
    int cond[3];
    certify(is, b_A, b_B, h, g, cond);
    if (!cond[0]) return fail(FM_E_UNCERTIFIED, "condition (i): a block sum of codes can leave int8");
    if (!cond[1]) return fail(FM_E_UNCERTIFIED, "condition (ii): a partial sum can leave int32");
    if (!cond[2]) return fail(FM_E_UNCERTIFIED, "condition (iii): a call spans two groups");
    // the kernel accumulates a whole group (all its calls) in int32
    if ((double)calls_per_group * is.LW * h * (is.LA * b_A) * (is.LB * b_B) >= 2147483648.0)
      return fail(FM_E_UNCERTIFIED, "a group's calls together can leave int32");
  }
  const int nc = is.gm * is.gn;
  for (int v : is.W)
    if (v < -1 || v > 1) return fail(FM_E_UNCERTIFIED, "combination weights must be -1, 0 or 1");
  const I8Layout L = i8_layout(is, M, N, K, h, corr);
  if (int rc = check_ws(workspace, ws_bytes, L.total)) return rc;
  char* ws = (char*)workspace;
  // host tables: coefficients per block (A: [r][i*gk + l], B: [r][j*gk + l],
  // rows zero-padded to coef_stride bytes) and the segments of every output
  // block (ascending r, padded)
  const int sa = coef_stride(is.gm * is.gk), sb = coef_stride(is.gn * is.gk);
  std::vector<int8_t> ca((size_t)is.R * sa, 0), cbt((size_t)is.R * sb, 0);
  for (int r = 0; r < is.R; ++r) {
    for (int i = 0; i < is.gm * is.gk; ++i) ca[(size_t)r * sa + i] = (int8_t)is.U[(size_t)r * is.gm * is.gk + i];
    for (int l = 0; l < is.gk; ++l)
      for (int j = 0; j < is.gn; ++j)
        cbt[(size_t)r * sb + j * is.gk + l] = (int8_t)is.V[(size_t)r * is.gk * is.gn + l * is.gn + j];
  }
  // segment entry: r | (w < 0) << 16 | (A side from the split parts q) << 17
  // | (B side from q) << 18; r = 0xffff pads a K step with zeros
  const int per_step = 128 / h;
  constexpr int32_t kNeg = 1 << 16, kQA = 1 << 17, kQB = 1 << 18;
  std::vector<int32_t> segs, off(1, 0), phase(2 * nc, -1);
  auto pad = [&]() {
    while ((segs.size() - off.back()) % per_step) segs.push_back(0xffff);
  };
  for (int c = 0; c < nc; ++c) {
    std::vector<int32_t> base;
    for (int r = 0; r < is.R; ++r) {
      const int w = is.W[(size_t)r * nc + c];
      if (w) base.push_back(r | (w < 0 ? kNeg : 0));
    }
    if (base.empty()) return fail(FM_E_ARG, "an output block combines no products");
    if (corr) {
      for (int32_t e : base) segs.push_back(e | kQA | kQB);  // R_A R_B
      pad();
      phase[2 * c] = (int32_t)(segs.size() - off.back()) / per_step;
      for (int32_t e : base) segs.push_back(e | kQA);  // R_A B0
      for (int32_t e : base) segs.push_back(e | kQB);  // A0 R_B
      pad();
      phase[2 * c + 1] = (int32_t)(segs.size() - off.back()) / per_step;
    }
    for (int32_t e : base) segs.push_back(e);  // A0 B0 (or the plain block sums)
    pad();
    off.push_back((int32_t)segs.size());
  }
  if ((int)segs.size() != L.nsegs) return fail(FM_E_ARG, "segment table size mismatch");
  // K steps of every output block's tiles, and their schedule
  std::vector<int> block_steps(nc);
  for (int c = 0; c < nc; ++c)
    block_steps[c] = (K / g) * calls_per_group * (off[c + 1] - off[c]) * h / 128;
  std::vector<int32_t> order, order_off;
  const int grid = i8_fast_schedule(is.gm, is.gn, M / is.gm, N / is.gn, block_steps, order, order_off);
  int rc = FM_OK;
  if ((rc = launch_fill_u32((uint32_t*)(ws + L.zero), kAlign / 4, 0u, st))) return rc;
  // the seven tables are adjacent in the workspace: one staged copy
  if ((rc = upload(ws + L.coefa,
                   {{ca.data(), ca.size()},
                    {cbt.data(), cbt.size()},
                    {segs.data(), segs.size() * 4},
                    {off.data(), off.size() * 4},
                    {order.data(), order.size() * 4},
                    {order_off.data(), order_off.size() * 4},
                    {phase.data(), phase.size() * 4}},
                   {0, L.coefb - L.coefa, L.segs - L.coefa, L.segoff - L.coefa,
                    L.order - L.coefa, L.order_off - L.coefa, L.phase - L.coefa},
                   L.phase - L.coefa + phase.size() * 4, st)))
    return rc;
  p.M = M;
  p.N = N;
  p.K = K;
  p.g = g;
  p.h = h;
  p.gm = is.gm;
  p.gn = is.gn;
  p.gk = is.gk;
  p.R = is.R;
  p.calls_per_group = calls_per_group;
  p.nsegs = (int)segs.size();
  p.grid = grid;
  p.sa = sa;
  p.sb = sb;
  p.corr = corr;
  p.qmax_a = qa;
  p.qmax_b = qb;
  p.ws = ws;
  p.ws_bytes = ws_bytes;
  p.flags = L.flags;
  p.zero = L.zero;
  p.coefa = L.coefa;
  p.coefb = L.coefb;
  p.segs = L.segs;
  p.segoff = L.segoff;
  p.order = L.order;
  p.order_off = L.order_off;
  p.phase = L.phase;
  p.t = L.t;
  p.s = L.s;
  p.sn = L.sn;
  p.tr = L.tr;
  p.sr = L.sr;
  p.snr = L.snr;
  return FM_OK;
}

// One fast call on a prepared workspace: block sums of A and B (split, with
// the correction), then the grouped products.
int i8_plan_run(const fm_int8_plan& p, const int8_t* Ac, const float* dA, const int8_t* BTc,
                const float* dB, float* out, hipStream_t st) {
  if (!Ac || !dA || !BTc || !dB || !out) return fail(FM_E_ARG, "null pointer");
  char* ws = p.ws;
  uint32_t* flag = (uint32_t*)(ws + p.flags);
  int8_t* T = (int8_t*)(ws + p.t);
  int8_t* S = (int8_t*)(ws + p.s);
  int8_t* Sn = (int8_t*)(ws + p.sn);
  int8_t* TR = p.corr ? (int8_t*)(ws + p.tr) : nullptr;
  int8_t* SR = p.corr ? (int8_t*)(ws + p.sr) : nullptr;
  int8_t* SnR = p.corr ? (int8_t*)(ws + p.snr) : nullptr;
  int rc = FM_OK;
  if ((rc = launch_fill_u32(flag, kAlign / 4, 0u, st))) return rc;
  if ((rc = launch_i8_form(Ac, p.M, p.K, p.gm, p.gk, p.h, p.R, (const int8_t*)(ws + p.coefa), p.sa,
                           T, nullptr, TR, nullptr, p.qmax_a, flag, st)))
    return rc;
  if ((rc = launch_i8_form(BTc, p.N, p.K, p.gn, p.gk, p.h, p.R, (const int8_t*)(ws + p.coefb), p.sb,
                           S, Sn, SR, SnR, p.qmax_b, flag, st)))
    return rc;
  return launch_i8_gemm(true, T, S, Sn, (const int8_t*)(ws + p.zero), dA, dB, out,
                        (const int32_t*)(ws + p.segs), (const int32_t*)(ws + p.segoff), p.nsegs,
                        (const int32_t*)(ws + p.order), (const int32_t*)(ws + p.order_off), p.grid,
                        p.M, p.N, p.K, p.g, p.gm, p.gn, p.R, p.h, p.calls_per_group, TR, SR, SnR,
                        p.corr ? (const int32_t*)(ws + p.phase) : nullptr, st);
}
}  // namespace

int fm_int8_certify(const fm_scheme* s, int levels, int b_A, int b_B, int h, int g,
                    int* conditions, double* L) try {
  clear_error();
  if (!conditions || !L) return fail(FM_E_ARG, "null pointer");
  IntScheme is;
  if (int rc = int_scheme(s, levels, is)) return rc;
  certify(is, b_A, b_B, h, g, conditions);
  L[0] = is.LA;
  L[1] = is.LB;
  L[2] = is.LW;
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_int8_certify_corrected(const fm_scheme* s, int levels, int b_A, int b_B, int h, int g,
                              int* conditions, double* bounds) try {
  clear_error();
  if (!conditions || !bounds) return fail(FM_E_ARG, "null pointer");
  IntScheme is;
  if (int rc = int_scheme(s, levels, is)) return rc;
  certify_corrected(is, b_A, b_B, h, g, conditions, bounds);
  return FM_OK;
} catch (...) {
  return host_failure();
}

size_t fm_int8_workspace_size(const fm_scheme* s, int levels, int M, int N, int K, int g, int h) try {
  IntScheme is;
  if (int_scheme(s, levels, is) != FM_OK) return 0;
  if (i8_fast_shape_ok(is, M, N, K, g, h) != FM_OK) return 0;
  return i8_layout(is, M, N, K, h, false).total;
} catch (...) {
  return host_failure(), (size_t)0;
}

size_t fm_int8_workspace_size_corrected(const fm_scheme* s, int levels, int M, int N, int K, int g,
                                        int h) try {
  IntScheme is;
  if (int_scheme(s, levels, is) != FM_OK) return 0;
  if (i8_fast_shape_ok(is, M, N, K, g, h) != FM_OK) return 0;
  return i8_layout(is, M, N, K, h, true).total;
} catch (...) {
  return host_failure(), (size_t)0;
}

int fm_int8_plan_create(const fm_scheme* s, int levels, int M, int N, int K, int g, int h,
                        int b_A, int b_B, int correct, void* workspace, size_t ws_bytes,
                        void* hip_stream, fm_int8_plan** out) try {
  clear_error();
  if (!out) return fail(FM_E_ARG, "null pointer");
  *out = nullptr;
  if (correct != 0 && correct != 1) return fail(FM_E_ARG, "correct must be 0 or 1");
  std::unique_ptr<fm_int8_plan> p(new (std::nothrow) fm_int8_plan());
  if (!p) return fail(FM_E_ARG, "out of host memory");
  if (int rc = i8_plan_prepare(s, levels, M, N, K, g, h, b_A, b_B, correct != 0, workspace,
                               ws_bytes, (hipStream_t)hip_stream, *p))
    return rc;
  *out = p.release();
  return FM_OK;
} catch (...) {
  return host_failure();
}

int fm_int8_plan_run(const fm_int8_plan* p, const int8_t* Ac, const float* dA, const int8_t* BTc,
                     const float* dB, float* out, void* hip_stream) try {
  clear_error();
  if (!p) return fail(FM_E_ARG, "null plan");
  return i8_plan_run(*p, Ac, dA, BTc, dB, out, (hipStream_t)hip_stream);
} catch (...) {
  return host_failure();
}

void fm_int8_plan_free(fm_int8_plan* p) { delete p; }

namespace {
int int8_fast_once(const fm_scheme* s, int levels, const int8_t* Ac, const float* dA,
                   const int8_t* BTc, const float* dB, int M, int N, int K, int g, int h, int b_A,
                   int b_B, bool corr, float* out, void* workspace, size_t ws_bytes,
                   void* hip_stream) {
  clear_error();
  if (!Ac || !dA || !BTc || !dB || !out) return fail(FM_E_ARG, "null pointer");
  fm_int8_plan p;
  hipStream_t st = (hipStream_t)hip_stream;
  if (int rc = i8_plan_prepare(s, levels, M, N, K, g, h, b_A, b_B, corr, workspace, ws_bytes, st,
                               p))
    return rc;
  return i8_plan_run(p, Ac, dA, BTc, dB, out, st);
}
}  // namespace

int fm_int8_matmul_fast(const fm_scheme* s, int levels, const int8_t* Ac, const float* dA,
                        const int8_t* BTc, const float* dB, int M, int N, int K, int g, int h,
                        int b_A, int b_B, float* out, void* workspace, size_t ws_bytes,
                        void* hip_stream) try {
  return int8_fast_once(s, levels, Ac, dA, BTc, dB, M, N, K, g, h, b_A, b_B, false, out,
                        workspace, ws_bytes, hip_stream);
} catch (...) {
  return host_failure();
}

int fm_int8_matmul_corrected(const fm_scheme* s, int levels, const int8_t* Ac, const float* dA,
                             const int8_t* BTc, const float* dB, int M, int N, int K, int g, int h,
                             int b_A, int b_B, float* out, void* workspace, size_t ws_bytes,
                             void* hip_stream) try {
  return int8_fast_once(s, levels, Ac, dA, BTc, dB, M, N, K, g, h, b_A, b_B, true, out,
                        workspace, ws_bytes, hip_stream);
} catch (...) {
  return host_failure();
}

}  // extern "C"

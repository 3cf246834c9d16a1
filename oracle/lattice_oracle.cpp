// Plain, slow CPU oracle for the permutohedral-lattice hot path of LatticeNet
// (Rosu, Schuett, Quenzel, Behnke, "LatticeNet: Fast Point Cloud
// Segmentation Using Permutohedral Lattices", arXiv:1912.05905).
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
// CPU-baseline leg of the benchmark may load this library.  It shares no code,
// header or constant with the GPU path.
//
// Design: std::map lattice keyed by integer coordinates, scalar loops,
// features accumulated in double.  Vertices are numbered in lexicographic
// key order (std::map order).  The embedding of a point (elevation, rounding,
// ranking, barycentric weights) is done in float32 with a fixed order of
// single roundings, because the vertex set it produces is a discontinuous
// function of that arithmetic; the paper fixes no precision for it.
//
// Sources followed:
//  * Notation: lattice V = (C, X), cloud P = (G, F), I_p, J_v (Notation).
//  * Lattice: projection of (d+1)Z^{d+1} along 1 onto H_d, coordinates sum
//    to zero, 2(d+1) neighbours at +-[-1..d..-1] (Permutohedral Lattice).
//  * Enclosing simplex by rounding: the paper defers to Baek and Adams; the
//    construction used is the closest-remainder-0-point / rank / sum-fix
//    method of Adams, Baek and Davis, "Fast High-Dimensional Filtering Using
//    the Permutohedral Lattice", Eurographics 2010, Sec. 3, restated here
//    from the mathematics.
//  * Scale G/sigma (Method), Splat Eq. (splat), Convolve (1-hop, missing
//    neighbour = 0, Fig. convolve), Slice Eq. (slice), Downsample and
//    Upsample (Proposed Operations), DeformSlice Eq. (deformSlice) with the
//    permutation-equivariant offset regressor.
//
// Readings of points the paper leaves open (each listed in the design notes):
//  * Elevation basis and scale: the isometric basis of H_d scaled by
//    (d+1)*sqrt(2/3), with fixed float32 operation order.
//  * Rounding ties go to the lower multiple of d+1; equal differentials rank
//    the lower coordinate index first.
//  * Simplex vertex k is the remainder-k vertex (consistent enumeration).
//  * Zero-weight vertices are inserted (|I_p| = d+1 always).
//  * Splat: sum of b*f, optionally divided by the sum of b (0/0 -> 0).
//  * Tap order 0 = self, 1..d+1 = +n_j, d+2..2d+2 = -n_j, n_j = (d+1)e_j - 1;
//    weights laid out W[tap][c_in][c_out].
//  * Coarse lattices come from the points with positions halved per level.
//  * Upsample: tap t of fine vertex f reads coarse vertex (f + o_t)/2 only
//    when that is a lattice point (all coordinates even and the halves
//    congruent mod d+1); every other tap, the centre included, is ignored.
//  * DeformSlice: max per channel over all d+1 weighted vertex values (the
//    vertex itself included), nonlinearity tanh.
//  * Distribute + PointNet: coordinates are the positions in lattice units
//    (g_p / sigma) minus their unweighted mean over J_v; three blocks of
//    GroupNorm, ReLU and a 1x1 layer, GroupNorm's statistics taken over all
//    distributed rows with one channel per group up to 32 channels and 32
//    groups above; then the per-vertex maximum.
//  * Group Normalization: statistics over all vertices of the lattice and the
//    group's channels, biased variance, eps inside the square root.
//  * Backward passes: gradients of the forward operators above; the ReLU's
//    derivative is 0 at 0 and DeformSlice's maximum passes its gradient to
//    the first maximal vertex, maximal among the float32 products b_k x_k.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <vector>

namespace {

constexpr int kDim = 3;              // d: dimension of the points
constexpr int kD1 = kDim + 1;        // d+1: lattice coordinates and simplex vertices
constexpr int kTaps = 2 * kD1 + 1;   // 1-hop neighbourhood incl. the centre
constexpr int32_t kCoordLimit = 1 << 20;

enum { OK = 0, EINVAL_ = -1, EUNSUPPORTED = -2, ENOMEM_ = -3, EHASHFULL = -4,
       EKEYRANGE = -5, ENONFINITE = -6, EDEVICE = -7, ELEVEL = -8 };

using Key = std::array<int32_t, kD1>;

struct Lattice {
  int64_t m = 0;
  int level = 0;
  std::vector<float> y;                 // m x (d+1) elevated positions (float32)
  std::map<Key, int64_t> index;         // key -> vertex number (lexicographic)
  std::vector<Key> keys;                // vertex number -> key
  std::vector<int64_t> idx;             // m x (d+1) simplex vertices of each point
  std::vector<float> bary;              // m x (d+1) barycentric weights
  const Lattice* parent = nullptr;      // finer lattice this one was coarsened from
  double scale[kDim] = {1.0, 1.0, 1.0}; // sigma_j * 2^level: positions in lattice units are g / scale
};

// ---------------------------------------------------------------------------
// Embedding of one point (float32, every line a single rounding).
// ---------------------------------------------------------------------------

// Per-axis factor a_j = s / (sigma_j * sqrt((j+1)(j+2))), s = (d+1) sqrt(2/3):
// scaling by 1/sigma (Method) folded into the isometric basis of H_d.
// Evaluated in double and rounded once to float32.
void axis_factors(const float* sigma, float a[kDim]) {
  const double s = (kDim + 1) * std::sqrt(2.0 / 3.0);
  for (int j = 0; j < kDim; ++j)
    a[j] = static_cast<float>(s / (static_cast<double>(sigma[j]) * std::sqrt(static_cast<double>((j + 1) * (j + 2)))));
}

// y = E (g / sigma) with E's columns orthonormal and orthogonal to 1, so
// y lies in H_d (coordinates sum to zero).  Column j of E has
// 1/sqrt((j+1)(j+2)) in rows 0..j and -(j+1)/sqrt((j+1)(j+2)) in row j+1.
void elevate(const float g[kDim], const float a[kDim], float y[kD1]) {
  float t[kDim];
  for (int j = 0; j < kDim; ++j) t[j] = g[j] * a[j];
  float run = 0.0f;                     // sum of t_j over j >= i
  for (int i = kDim; i >= 1; --i) {
    const float it = static_cast<float>(i) * t[i - 1];
    y[i] = run - it;
    run = run + t[i - 1];
  }
  y[0] = run;
}

// Enclosing simplex of y: the d+1 vertex keys (vertex k has every coordinate
// congruent to k mod d+1) and the barycentric weights b_k.
void enclosing_simplex(const float y[kD1], Key vert[kD1], float b[kD1]) {
  const float inv = 1.0f / static_cast<float>(kD1);   // exact for d = 3
  const float step = static_cast<float>(kD1);
  // nearest point of (d+1)Z per coordinate; a tie goes to the lower one
  int32_t base[kD1];
  int32_t total = 0;
  for (int i = 0; i < kD1; ++i) {
    const float lo = std::floor(y[i] * inv) * step;
    const float hi = lo + step;
    const float up = hi - y[i];
    const float down = y[i] - lo;
    base[i] = static_cast<int32_t>(up < down ? hi : lo);
    total += base[i];
  }
  const int32_t excess = total / kD1;  // base lies on H_d iff excess == 0
  float diff[kD1];
  for (int i = 0; i < kD1; ++i) diff[i] = y[i] - static_cast<float>(base[i]);
  // rank: 0 for the largest differential; ties rank the lower index first
  int rank[kD1];
  for (int i = 0; i < kD1; ++i) {
    rank[i] = 0;
    for (int j = 0; j < kD1; ++j)
      if (diff[j] > diff[i] || (diff[j] == diff[i] && j < i)) ++rank[i];
  }
  // move base onto H_d: shift the |excess| coordinates whose differentials
  // are most extreme by d+1, which rotates the ranks
  if (excess > 0) {
    for (int i = 0; i < kD1; ++i) {
      if (rank[i] >= kD1 - excess) { base[i] -= kD1; rank[i] += excess - kD1; }
      else rank[i] += excess;
    }
  } else if (excess < 0) {
    for (int i = 0; i < kD1; ++i) {
      if (rank[i] < -excess) { base[i] += kD1; rank[i] += kD1 + excess; }
      else rank[i] += excess;
    }
  }
  // sorted scaled differentials z_0 >= ... >= z_d
  float z[kD1];
  for (int i = 0; i < kD1; ++i) z[rank[i]] = (y[i] - static_cast<float>(base[i])) * inv;
  b[0] = 1.0f - (z[0] - z[kDim]);
  for (int k = 1; k < kD1; ++k) b[k] = z[kDim - k] - z[kDim - k + 1];
  // vertex k: base + k*1, minus (d+1) on the k coordinates of smallest
  // differential (the k highest ranks)
  for (int k = 0; k < kD1; ++k)
    for (int i = 0; i < kD1; ++i)
      vert[k][i] = base[i] + k - (rank[i] > kDim - k ? kD1 : 0);
}

bool key_in_range(const Key& c) {
  for (int i = 0; i < kD1; ++i)
    if (c[i] >= kCoordLimit || c[i] <= -kCoordLimit) return false;
  return true;
}

// Offsets of the 1-hop taps: o_0 = 0, o_{1+j} = +n_j, o_{d+2+j} = -n_j,
// with n_j = (d+1) e_j - 1.
Key tap_offset(int t) {
  Key o{};
  if (t == 0) return o;
  const int j = (t - 1) % kD1;
  const int sign = t <= kD1 ? 1 : -1;
  for (int i = 0; i < kD1; ++i) o[i] = sign * ((i == j ? kD1 : 0) - 1);
  return o;
}

// Build the lattice of m points given their elevated positions.
int build_from_elevated(Lattice* L) {
  const int64_t m = L->m;
  std::vector<Key> pv(static_cast<size_t>(m) * kD1);
  L->bary.assign(static_cast<size_t>(m) * kD1, 0.0f);
  for (int64_t p = 0; p < m; ++p) {
    const float* y = &L->y[static_cast<size_t>(p) * kD1];
    for (int i = 0; i < kD1; ++i) {
      if (!std::isfinite(y[i])) return ENONFINITE;
      if (std::fabs(y[i]) >= 2.0f * kCoordLimit) return EKEYRANGE;  // keys would leave the range
    }
    enclosing_simplex(y, &pv[static_cast<size_t>(p) * kD1], &L->bary[static_cast<size_t>(p) * kD1]);
    for (int k = 0; k < kD1; ++k) {
      const Key& c = pv[static_cast<size_t>(p) * kD1 + k];
      if (!key_in_range(c)) return EKEYRANGE;
      L->index.emplace(c, 0);
    }
  }
  int64_t next = 0;
  L->keys.reserve(L->index.size());
  for (auto& kv : L->index) { kv.second = next++; L->keys.push_back(kv.first); }
  L->idx.resize(static_cast<size_t>(m) * kD1);
  for (size_t e = 0; e < pv.size(); ++e) L->idx[e] = L->index.at(pv[e]);
  return OK;
}

int64_t find_vertex(const Lattice* L, const Key& c) {
  if (!key_in_range(c)) return -1;
  auto it = L->index.find(c);
  return it == L->index.end() ? -1 : it->second;
}

// Neighbour table of a lattice (n x taps); -1 = vertex not allocated.
std::vector<int64_t> same_level_table(const Lattice* L) {
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::vector<int64_t> nb(static_cast<size_t>(n) * kTaps);
  for (int64_t v = 0; v < n; ++v)
    for (int t = 0; t < kTaps; ++t) {
      Key c = L->keys[v];
      const Key o = tap_offset(t);
      for (int i = 0; i < kD1; ++i) c[i] += o[i];
      nb[static_cast<size_t>(v) * kTaps + t] = find_vertex(L, c);
    }
  return nb;
}

// Downsample: coarse vertex c reads the fine vertices at 2c + o_t (the coarse
// lattice embedded in the fine one by scaling by 2).
std::vector<int64_t> down_table(const Lattice* coarse, const Lattice* fine) {
  const int64_t n = static_cast<int64_t>(coarse->keys.size());
  std::vector<int64_t> nb(static_cast<size_t>(n) * kTaps);
  for (int64_t v = 0; v < n; ++v)
    for (int t = 0; t < kTaps; ++t) {
      Key c = coarse->keys[v];
      const Key o = tap_offset(t);
      for (int i = 0; i < kD1; ++i) c[i] = 2 * c[i] + o[i];
      nb[static_cast<size_t>(v) * kTaps + t] = find_vertex(fine, c);
    }
  return nb;
}

// Upsample: fine vertex f reads the coarse vertex (f + o_t)/2 when that is a
// lattice point; fractional neighbours contribute nothing.
std::vector<int64_t> up_table(const Lattice* fine, const Lattice* coarse) {
  const int64_t n = static_cast<int64_t>(fine->keys.size());
  std::vector<int64_t> nb(static_cast<size_t>(n) * kTaps);
  for (int64_t v = 0; v < n; ++v)
    for (int t = 0; t < kTaps; ++t) {
      Key u = fine->keys[v];
      const Key o = tap_offset(t);
      bool lattice_point = true;
      for (int i = 0; i < kD1; ++i) {
        u[i] += o[i];
        if (u[i] % 2 != 0) lattice_point = false;
      }
      int64_t found = -1;
      if (lattice_point) {
        Key h;
        for (int i = 0; i < kD1; ++i) h[i] = u[i] / 2;
        const int r0 = ((h[0] % kD1) + kD1) % kD1;
        for (int i = 1; i < kD1; ++i)
          if (((h[i] % kD1) + kD1) % kD1 != r0) lattice_point = false;
        if (lattice_point) found = find_vertex(coarse, h);
      }
      nb[static_cast<size_t>(v) * kTaps + t] = found;
    }
  return nb;
}

// Y[v] = bias + sum_t sum_c X[nb[v][t]][c] W[t][c][:], missing taps add 0.
void conv_with_table(const std::vector<int64_t>& nb, const double* X, int64_t ldx, int cin,
                     const double* W, const double* bias, int cout, int relu,
                     const int64_t* rows, int64_t nrows, double* Y, int64_t ldy) {
  std::vector<double> acc(cout);
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t v = rows ? rows[r] : r;
    for (int o = 0; o < cout; ++o) acc[o] = bias ? bias[o] : 0.0;
    for (int t = 0; t < kTaps; ++t) {
      const int64_t u = nb[static_cast<size_t>(v) * kTaps + t];
      if (u < 0) continue;
      for (int c = 0; c < cin; ++c) {
        const double x = X[u * ldx + c];
        const double* wrow = W + (static_cast<int64_t>(t) * cin + c) * cout;
        for (int o = 0; o < cout; ++o) acc[o] += x * wrow[o];
      }
    }
    for (int o = 0; o < cout; ++o) {
      double val = acc[o];
      if (relu && val < 0.0) val = 0.0;
      Y[r * ldy + o] = val;
    }
  }
}

}  // namespace

extern "C" {

typedef struct Lattice orc_lattice;

// Per-axis elevation factors (for pins).
void orc_axis_factors(const float* sigma, float* a) { axis_factors(sigma, a); }

// Elevate m points: pos m x d, sigma d -> y m x (d+1).
int orc_elevate(const float* pos, int64_t m, const float* sigma, float* y) {
  if (!pos || !sigma || !y || m < 0) return EINVAL_;
  float a[kDim];
  axis_factors(sigma, a);
  for (int64_t p = 0; p < m; ++p) elevate(pos + p * kDim, a, y + p * kD1);
  return OK;
}

// Enclosing simplices of m elevated points: keys m x (d+1) x (d+1), w m x (d+1).
int orc_simplex(const float* y, int64_t m, int32_t* keys, float* w) {
  if (!y || !keys || !w || m < 0) return EINVAL_;
  for (int64_t p = 0; p < m; ++p) {
    Key vert[kD1];
    enclosing_simplex(y + p * kD1, vert, w + p * kD1);
    for (int k = 0; k < kD1; ++k)
      for (int i = 0; i < kD1; ++i) keys[(p * kD1 + k) * kD1 + i] = vert[k][i];
  }
  return OK;
}

// Lattice of a cloud: positions m x d (float32), sigma d.
int orc_create(const float* pos, int64_t m, int d, const float* sigma, orc_lattice** out) {
  if (!out) return EINVAL_;
  *out = nullptr;
  if (d != kDim) return EUNSUPPORTED;
  if (m < 0 || (m > 0 && !pos) || !sigma) return EINVAL_;
  for (int j = 0; j < kDim; ++j)
    if (!(sigma[j] > 0.0f) || !std::isfinite(sigma[j])) return EINVAL_;
  for (int64_t e = 0; e < m * kDim; ++e)
    if (!std::isfinite(pos[e])) return ENONFINITE;
  Lattice* L = new Lattice();
  L->m = m;
  for (int j = 0; j < kDim; ++j) L->scale[j] = sigma[j];
  L->y.resize(static_cast<size_t>(m) * kD1);
  orc_elevate(pos, m, sigma, L->y.data());
  const int st = build_from_elevated(L);
  if (st != OK) { delete L; return st; }
  *out = L;
  return OK;
}

// Next-coarser lattice: the same points with elevated positions halved
// (equivalently, positions divided by 2).
int orc_coarsen(const orc_lattice* fine, orc_lattice** out) {
  if (!fine || !out) return EINVAL_;
  Lattice* L = new Lattice();
  L->m = fine->m;
  L->level = fine->level + 1;
  L->parent = fine;
  for (int j = 0; j < kDim; ++j) L->scale[j] = 2.0 * fine->scale[j];
  L->y.resize(fine->y.size());
  for (size_t e = 0; e < fine->y.size(); ++e) L->y[e] = fine->y[e] * 0.5f;
  const int st = build_from_elevated(L);
  if (st != OK) { delete L; return st; }
  *out = L;
  return OK;
}

void orc_destroy(orc_lattice* L) { delete L; }
int64_t orc_num_vertices(const orc_lattice* L) { return static_cast<int64_t>(L->keys.size()); }
int64_t orc_num_points(const orc_lattice* L) { return L->m; }
int orc_level(const orc_lattice* L) { return L->level; }

void orc_export_elevated(const orc_lattice* L, float* y) {
  std::memcpy(y, L->y.data(), L->y.size() * sizeof(float));
}

void orc_export_keys(const orc_lattice* L, int32_t* keys) {
  for (size_t v = 0; v < L->keys.size(); ++v)
    for (int i = 0; i < kD1; ++i) keys[v * kD1 + i] = L->keys[v][i];
}

void orc_export_simplices(const orc_lattice* L, int64_t* idx, float* w) {
  std::memcpy(idx, L->idx.data(), L->idx.size() * sizeof(int64_t));
  std::memcpy(w, L->bary.data(), L->bary.size() * sizeof(float));
}

void orc_export_neighbors(const orc_lattice* L, int64_t* nbr) {
  const auto nb = same_level_table(L);
  std::memcpy(nbr, nb.data(), nb.size() * sizeof(int64_t));
}

void orc_export_down_table(const orc_lattice* coarse, int64_t* nbr) {
  const auto nb = down_table(coarse, coarse->parent);
  std::memcpy(nbr, nb.data(), nb.size() * sizeof(int64_t));
}

void orc_export_up_table(const orc_lattice* coarse, int64_t* nbr) {
  const auto nb = up_table(coarse->parent, coarse);
  std::memcpy(nbr, nb.data(), nb.size() * sizeof(int64_t));
}

// Splat, Eq. (splat): x_v = sum_{p in J_v} b_pv f_p; wsum_v = sum b_pv.
// normalize != 0 divides by wsum (weighted average), 0 where wsum == 0.
int orc_splat(const orc_lattice* L, const double* F, int C, int normalize, double* X, double* wsum) {
  if (!L || C <= 0 || (L->m > 0 && !F) || !X) return EINVAL_;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::vector<double> ws(n, 0.0);
  std::fill(X, X + n * C, 0.0);
  for (int64_t p = 0; p < L->m; ++p)
    for (int k = 0; k < kD1; ++k) {
      const int64_t v = L->idx[p * kD1 + k];
      const double b = L->bary[p * kD1 + k];
      ws[v] += b;
      for (int c = 0; c < C; ++c) X[v * C + c] += b * F[p * C + c];
    }
  if (normalize)
    for (int64_t v = 0; v < n; ++v)
      for (int c = 0; c < C; ++c) X[v * C + c] = ws[v] > 0.0 ? X[v * C + c] / ws[v] : 0.0;
  if (wsum) std::copy(ws.begin(), ws.end(), wsum);
  return OK;
}

// Convolution.  dst == src: 1-hop convolution over the 2(d+1)+1 vertices.
// dst coarsened from src: strided convolution (Downsample).  rows (optional)
// selects the output vertices computed; Y then holds nrows rows.
int orc_conv(const orc_lattice* dst, const orc_lattice* src, const double* X, int64_t ldx, int cin,
             const double* W, const double* bias, int cout, int relu,
             const int64_t* rows, int64_t nrows, double* Y, int64_t ldy) {
  if (!dst || !src || !X || !W || !Y || cin <= 0 || cout <= 0) return EINVAL_;
  std::vector<int64_t> nb;
  if (dst == src) nb = same_level_table(dst);
  else if (dst->parent == src) nb = down_table(dst, src);
  else return ELEVEL;
  if (!rows) nrows = static_cast<int64_t>(dst->keys.size());
  conv_with_table(nb, X, ldx, cin, W, bias, cout, relu, rows, nrows, Y, ldy);
  return OK;
}

// Upsample (transposed convolution) from coarse to its parent fine lattice.
int orc_refine(const orc_lattice* fine, const orc_lattice* coarse, const double* X, int64_t ldx, int cin,
               const double* W, const double* bias, int cout, int relu,
               const int64_t* rows, int64_t nrows, double* Y, int64_t ldy) {
  if (!fine || !coarse || !X || !W || !Y || cin <= 0 || cout <= 0) return EINVAL_;
  if (coarse->parent != fine) return ELEVEL;
  const auto nb = up_table(fine, coarse);
  if (!rows) nrows = static_cast<int64_t>(fine->keys.size());
  conv_with_table(nb, X, ldx, cin, W, bias, cout, relu, rows, nrows, Y, ldy);
  return OK;
}

// Slice, Eq. (slice), on explicit simplices: out_p = sum_k w_pk X[idx_pk].
void orc_slice_raw(const double* X, int64_t ldx, int C, const int64_t* idx, const float* w,
                   int64_t m, const int64_t* pts, double* out) {
  for (int64_t r = 0; r < m; ++r) {
    const int64_t p = pts ? pts[r] : r;
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int k = 0; k < kD1; ++k)
        acc += static_cast<double>(w[p * kD1 + k]) * X[idx[p * kD1 + k] * ldx + c];
      out[r * C + c] = acc;
    }
  }
}

// DeformSlice, Eq. (deformSlice) with the equivariant offset regressor:
//   q_k = b_k x_k,  M = max_k q_k (per channel),
//   db_k = tanh(beta + (q_k - M) . wv),  out = sum_k (b_k + db_k) x_k.
void orc_deform_slice_raw(const double* X, int64_t ldx, int C, const int64_t* idx, const float* w,
                          int64_t m, const double* wv, double beta, const int64_t* pts,
                          double* out, double* delta) {
  std::vector<double> q(static_cast<size_t>(kD1) * C), mx(C);
  for (int64_t r = 0; r < m; ++r) {
    const int64_t p = pts ? pts[r] : r;
    for (int k = 0; k < kD1; ++k)
      for (int c = 0; c < C; ++c)
        q[k * C + c] = static_cast<double>(w[p * kD1 + k]) * X[idx[p * kD1 + k] * ldx + c];
    for (int c = 0; c < C; ++c) {
      mx[c] = q[c];
      for (int k = 1; k < kD1; ++k) mx[c] = std::max(mx[c], q[k * C + c]);
    }
    double db[kD1];
    for (int k = 0; k < kD1; ++k) {
      double s = beta;
      for (int c = 0; c < C; ++c) s += (q[k * C + c] - mx[c]) * wv[c];
      db[k] = std::tanh(s);
      if (delta) delta[r * kD1 + k] = db[k];
    }
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int k = 0; k < kD1; ++k)
        acc += (static_cast<double>(w[p * kD1 + k]) + db[k]) * X[idx[p * kD1 + k] * ldx + c];
      out[r * C + c] = acc;
    }
  }
}

// DeformSlice fused with the last linear classification layer
// (Implementation): logits_p = Wc f_p + bc with f_p the DeformSlice output
// of point p, Wc laid out [class][channel] (K x C), bc optional.
int orc_deform_slice_classify(const orc_lattice* L, const double* X, int64_t ldx, int C, const double* wv,
                              double beta, const double* Wc, const double* bc, int K, double* logits) {
  if (!L || !X || !wv || !Wc || !logits || C <= 0 || K <= 0) return EINVAL_;
  std::vector<double> f(static_cast<size_t>(L->m) * C);
  orc_deform_slice_raw(X, ldx, C, L->idx.data(), L->bary.data(), L->m, wv, beta, nullptr, f.data(), nullptr);
  for (int64_t p = 0; p < L->m; ++p)
    for (int j = 0; j < K; ++j) {
      double a = bc ? bc[j] : 0.0;
      for (int c = 0; c < C; ++c) a += Wc[static_cast<int64_t>(j) * C + c] * f[p * C + c];
      logits[p * K + j] = a;
    }
  return OK;
}

int orc_slice(const orc_lattice* L, const double* X, int64_t ldx, int C,
              const int64_t* pts, int64_t npts, double* out) {
  if (!L || !X || !out || C <= 0) return EINVAL_;
  orc_slice_raw(X, ldx, C, L->idx.data(), L->bary.data(), pts ? npts : L->m, pts, out);
  return OK;
}

int orc_deform_slice(const orc_lattice* L, const double* X, int64_t ldx, int C, const double* wv,
                     double beta, const int64_t* pts, int64_t npts, double* out, double* delta) {
  if (!L || !X || !out || !wv || C <= 0) return EINVAL_;
  orc_deform_slice_raw(X, ldx, C, L->idx.data(), L->bary.data(), pts ? npts : L->m, wv, beta,
                       pts, out, delta);
  return OK;
}

// Distribute + PointNet (Proposed Operations, Eq. (distribute), and the
// PointNet block of the architecture figure).
//  * Distribute: every vertex v receives one row per point p of J_v (the
//    points whose simplex contains v), r = [g_p - mu_v ; f_p], where g_p are
//    the positions in lattice units (G_s = G / sigma of the Method section,
//    sigma doubled per coarsening level) and mu_v is the mean of g_p over J_v.
//  * PointNet: three blocks [GroupNorm, ReLU, 1x1], h_i = W_i relu(GN_i(h_{i-1})) + b_i
//    (h_0 = r, W_i laid out [out][in]), then x_v = the per-channel maximum
//    of h_3 over the rows of v (MaxPool).
//  * GroupNorm over the whole set of distributed rows (all (v, p) pairs) and
//    the channels of a group; a layer of C <= 32 channels has one channel
//    per group, a wider one 32 groups (C a multiple of 32).  gamma / beta
//    hold the per-channel affine parameters of the three normalisations one
//    after the other ((d + Cf) + C1 + C2 values each); null means 1 / 0.
// G is m x d raw positions, F m x Cf features; X gets n x C3.  Plain loops in
// double over the distributed-row matrix; a NaN anywhere propagates to the
// outputs (the ReLU and the maximum keep NaN).
int orc_groupnorm(const double* X, int64_t n, int C, int64_t ldx, int groups, const double* gamma,
                  const double* beta, double eps, int relu, double* Y, int64_t ldy);

int orc_distribute_pointnet(const orc_lattice* L, const double* G, const double* F, int cf, const double* gamma,
                            const double* beta, double eps, const double* W1, const double* b1, int c1,
                            const double* W2, const double* b2, int c2, const double* W3, const double* b3, int c3,
                            double* X) {
  if (!L || !X || cf < 0 || c1 <= 0 || c2 <= 0 || c3 <= 0 || !W1 || !W2 || !W3 || !(eps >= 0.0)) return EINVAL_;
  if (L->m > 0 && (!G || (cf > 0 && !F))) return EINVAL_;
  const int cin = kDim + cf;
  const int widths[3] = {cin, c1, c2};
  for (int w : widths)
    if (w > 32 && w % 32 != 0) return EUNSUPPORTED;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  // J_v: the points whose simplex has v among its d+1 vertices
  std::vector<std::vector<int64_t>> J(n);
  for (int64_t p = 0; p < L->m; ++p)
    for (int k = 0; k < kD1; ++k) J[L->idx[p * kD1 + k]].push_back(p);
  // the distributed rows, vertex by vertex
  const int64_t rows = L->m * kD1;
  std::vector<int64_t> row_vertex;
  row_vertex.reserve(rows);
  std::vector<double> h(static_cast<size_t>(rows) * cin);
  int64_t r = 0;
  for (int64_t v = 0; v < n; ++v) {
    double mu[kDim] = {0.0, 0.0, 0.0};
    for (int64_t p : J[v])
      for (int j = 0; j < kDim; ++j) mu[j] += G[p * kDim + j] / L->scale[j];
    for (int j = 0; j < kDim; ++j) mu[j] /= static_cast<double>(J[v].size());
    for (int64_t p : J[v]) {
      for (int j = 0; j < kDim; ++j) h[r * cin + j] = G[p * kDim + j] / L->scale[j] - mu[j];
      for (int c = 0; c < cf; ++c) h[r * cin + kDim + c] = F[p * cf + c];
      row_vertex.push_back(v);
      ++r;
    }
  }
  // three [GN, ReLU, 1x1] blocks
  const double* Ws[3] = {W1, W2, W3};
  const double* bs[3] = {b1, b2, b3};
  const int outs[3] = {c1, c2, c3};
  int off = 0;   // first affine parameter of the current normalisation
  for (int layer = 0; layer < 3; ++layer) {
    const int ci = widths[layer], co = outs[layer];
    const int groups = ci <= 32 ? ci : 32;
    std::vector<double> a(h.size());
    if (rows > 0) {
      const int st = orc_groupnorm(h.data(), rows, ci, ci, groups, gamma ? gamma + off : nullptr,
                                   beta ? beta + off : nullptr, eps, 1, a.data(), ci);
      if (st != OK) return st;
    }
    off += ci;
    std::vector<double> next(static_cast<size_t>(rows) * co);
    for (int64_t q = 0; q < rows; ++q)
      for (int o = 0; o < co; ++o) {
        double acc = bs[layer] ? bs[layer][o] : 0.0;
        for (int i = 0; i < ci; ++i) acc += Ws[layer][o * ci + i] * a[q * ci + i];
        next[q * co + o] = acc;
      }
    h.swap(next);
  }
  // MaxPool over the rows of each vertex (NaN wins)
  for (int64_t e = 0; e < n * c3; ++e) X[e] = -INFINITY;
  for (int64_t q = 0; q < rows; ++q) {
    double* x = X + row_vertex[q] * c3;
    for (int o = 0; o < c3; ++o) {
      const double val = h[q * c3 + o];
      if (std::isnan(x[o])) continue;
      if (std::isnan(val) || val > x[o]) x[o] = val;
    }
  }
  return OK;
}

// ---------------------------------------------------------------------------
// Backward passes (Implementation: the lattice operators have forward and
// backward passes on the GPU).  Each is the gradient of its forward operator
// for a scalar loss L with dL/d(output) given; for the linear operators that
// is the adjoint.  Written from the definitions, point by point / vertex by
// vertex.
// ---------------------------------------------------------------------------

// Splat backward: dF_p = sum_{v in I_p} b_pv dX_v, each term divided by
// wsum_v = sum_{q in J_v} b_qv when the forward normalised (0 where wsum_v is
// 0, as in the forward).
int orc_splat_backward(const orc_lattice* L, const double* dX, int C, int normalize, double* dF) {
  if (!L || C <= 0 || !dX || (L->m > 0 && !dF)) return EINVAL_;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::vector<double> ws(n, 0.0);
  for (int64_t p = 0; p < L->m; ++p)
    for (int k = 0; k < kD1; ++k) ws[L->idx[p * kD1 + k]] += L->bary[p * kD1 + k];
  for (int64_t p = 0; p < L->m; ++p)
    for (int c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int k = 0; k < kD1; ++k) {
        const int64_t v = L->idx[p * kD1 + k];
        double coef = L->bary[p * kD1 + k];
        if (normalize) coef = ws[v] > 0.0 ? coef / ws[v] : 0.0;
        acc += coef * dX[v * C + c];
      }
      dF[p * C + c] = acc;
    }
  return OK;
}

// Slice backward: dX_v = sum over the pairs (p, k) with I_p[k] = v of
// b_pk dOut_p.
int orc_slice_backward(const orc_lattice* L, const double* dOut, int C, double* dX) {
  if (!L || C <= 0 || !dX || (L->m > 0 && !dOut)) return EINVAL_;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::fill(dX, dX + n * C, 0.0);
  for (int64_t p = 0; p < L->m; ++p)
    for (int k = 0; k < kD1; ++k) {
      const int64_t v = L->idx[p * kD1 + k];
      const double b = L->bary[p * kD1 + k];
      for (int c = 0; c < C; ++c) dX[v * C + c] += b * dOut[p * C + c];
    }
  return OK;
}

// Convolution backward for the three forms: dst == src (1-hop), dst coarsened
// from src (strided), src coarsened from dst (Upsample into dst).  The
// forward was Y_v = act(bias + sum_t X[nb(v,t)] W[t]) with W[t] laid out
// [c_in][c_out]; with G = dY, masked by Y > 0 when act is the ReLU (the
// derivative taken as 0 at 0):
//   dX[nb(v,t)] += W[t] G_v,  dW[t] += X[nb(v,t)]^T G_v,  dbias += G_v.
// Any of dX, dW, dbias may be null.  dX is n_src x cin, dW taps x cin x cout.
int orc_conv_backward(const orc_lattice* dst, const orc_lattice* src, const double* X, int cin,
                      const double* W, int cout, int relu, const double* Y, const double* dY,
                      double* dX, double* dW, double* dbias) {
  if (!dst || !src || !dY || cin <= 0 || cout <= 0 || (relu && !Y)) return EINVAL_;
  if ((dX && !W) || (dW && !X)) return EINVAL_;
  std::vector<int64_t> nb;
  if (dst == src) nb = same_level_table(dst);
  else if (dst->parent == src) nb = down_table(dst, src);
  else if (src->parent == dst) nb = up_table(dst, src);
  else return ELEVEL;
  const int64_t n_out = static_cast<int64_t>(dst->keys.size());
  const int64_t n_in = static_cast<int64_t>(src->keys.size());
  if (dX) std::fill(dX, dX + n_in * cin, 0.0);
  if (dW) std::fill(dW, dW + static_cast<int64_t>(kTaps) * cin * cout, 0.0);
  if (dbias) std::fill(dbias, dbias + cout, 0.0);
  std::vector<double> g(cout);
  for (int64_t v = 0; v < n_out; ++v) {
    for (int o = 0; o < cout; ++o) {
      g[o] = dY[v * cout + o];
      if (relu && !(Y[v * cout + o] > 0.0)) g[o] = 0.0;
      if (dbias) dbias[o] += g[o];
    }
    for (int t = 0; t < kTaps; ++t) {
      const int64_t u = nb[static_cast<size_t>(v) * kTaps + t];
      if (u < 0) continue;
      for (int c = 0; c < cin; ++c) {
        const int64_t wrow = (static_cast<int64_t>(t) * cin + c) * cout;
        if (dX) {
          double a = 0.0;
          for (int o = 0; o < cout; ++o) a += W[wrow + o] * g[o];
          dX[u * cin + c] += a;
        }
        if (dW)
          for (int o = 0; o < cout; ++o) dW[wrow + o] += X[u * cin + c] * g[o];
      }
    }
  }
  return OK;
}

// DeformSlice backward.  Forward per point p (vertex k of its simplex, value
// x_k = X[I_p[k]], weight b_k):
//   q_k = b_k x_k,  M = max_k q_k per channel (at the first k maximal in float32),
//   s_k = beta + (q_k - M) . wv,  db_k = tanh(s_k),  out = sum_k (b_k + db_k) x_k.
// With g = dOut_p, a_k = g . x_k and e_k = a_k (1 - db_k^2) = dL/ds_k:
//   dx_k += (b_k + db_k) g + e_k b_k wv - [k = argmax_c] (sum_j e_j) b_k wv_c,
//   dwv  += sum_k e_k (q_k - M),   dbeta += sum_k e_k.
int orc_deform_slice_backward(const orc_lattice* L, const double* X, int C, const double* wv, double beta,
                              const double* dOut, double* dX, double* dwv, double* dbeta) {
  if (!L || !X || !wv || C <= 0 || !dX || !dwv || !dbeta || (L->m > 0 && !dOut)) return EINVAL_;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::fill(dX, dX + n * C, 0.0);
  std::fill(dwv, dwv + C, 0.0);
  *dbeta = 0.0;
  std::vector<double> q(static_cast<size_t>(kD1) * C), mx(C);
  std::vector<int> am(C);
  for (int64_t p = 0; p < L->m; ++p) {
    const int64_t* I = &L->idx[p * kD1];
    const float* b = &L->bary[p * kD1];
    for (int k = 0; k < kD1; ++k)
      for (int c = 0; c < C; ++c) q[k * C + c] = static_cast<double>(b[k]) * X[I[k] * C + c];
    // the vertex that receives the maximum's gradient is decided on the
    // float32 products b_k x_k (the GPU's precision): a discrete choice taken
    // by floating point must be taken the same way on both sides
    for (int c = 0; c < C; ++c) {
      am[c] = 0;
      float best = static_cast<float>(b[0]) * static_cast<float>(X[I[0] * C + c]);
      for (int k = 1; k < kD1; ++k) {
        const float qk = static_cast<float>(b[k]) * static_cast<float>(X[I[k] * C + c]);
        if (qk > best) {
          best = qk;
          am[c] = k;
        }
      }
      mx[c] = q[am[c] * C + c];
    }
    const double* g = dOut + p * C;
    double db[kD1], e[kD1], esum = 0.0;
    for (int k = 0; k < kD1; ++k) {
      double sk = beta, ak = 0.0;
      for (int c = 0; c < C; ++c) {
        sk += (q[k * C + c] - mx[c]) * wv[c];
        ak += g[c] * X[I[k] * C + c];
      }
      db[k] = std::tanh(sk);
      e[k] = ak * (1.0 - db[k] * db[k]);
      esum += e[k];
    }
    for (int k = 0; k < kD1; ++k)
      for (int c = 0; c < C; ++c) {
        double d = (static_cast<double>(b[k]) + db[k]) * g[c] + e[k] * b[k] * wv[c];
        if (am[c] == k) d -= esum * b[k] * wv[c];
        dX[I[k] * C + c] += d;
      }
    for (int k = 0; k < kD1; ++k) {
      for (int c = 0; c < C; ++c) dwv[c] += e[k] * (q[k * C + c] - mx[c]);
      *dbeta += e[k];
    }
  }
  return OK;
}

// Group Normalization (Implementation: every convolution is pre-activated
// by Group Normalization with 32 groups and a ReLU; Wu and He, "Group
// Normalization", ECCV 2018), over the vertices of one lattice: channel c
// belongs to group c / (C / groups); each group's mean and (biased)
// variance are taken over all n rows and its channels; then
//   Y[v][c] = (X[v][c] - mean_g) / sqrt(var_g + eps) * gamma_c + beta_c,
// followed by max(., 0) when relu != 0.  gamma / beta null mean 1 / 0.
int orc_groupnorm(const double* X, int64_t n, int C, int64_t ldx, int groups, const double* gamma,
                  const double* beta, double eps, int relu, double* Y, int64_t ldy) {
  if (!X || !Y || n < 0 || C <= 0 || groups <= 0 || C % groups != 0 || !(eps >= 0.0)) return EINVAL_;
  const int per = C / groups;
  for (int g = 0; g < groups; ++g) {
    double mean = 0.0;
    for (int64_t v = 0; v < n; ++v)
      for (int c = g * per; c < (g + 1) * per; ++c) mean += X[v * ldx + c];
    const double cnt = static_cast<double>(n) * per;
    mean = cnt > 0 ? mean / cnt : 0.0;
    double var = 0.0;
    for (int64_t v = 0; v < n; ++v)
      for (int c = g * per; c < (g + 1) * per; ++c) var += (X[v * ldx + c] - mean) * (X[v * ldx + c] - mean);
    var = cnt > 0 ? var / cnt : 0.0;
    const double inv = 1.0 / std::sqrt(var + eps);
    for (int64_t v = 0; v < n; ++v)
      for (int c = g * per; c < (g + 1) * per; ++c) {
        double y = (X[v * ldx + c] - mean) * inv * (gamma ? gamma[c] : 1.0) + (beta ? beta[c] : 0.0);
        if (relu && y < 0.0) y = 0.0;
        Y[v * ldy + c] = y;
      }
  }
  return OK;
}

// Group Normalization backward: the gradient of orc_groupnorm for a scalar
// loss with dL/dY = dY (n x C, dense), written from the forward's definition.
// Per group g (N = n * C / groups values), xhat = (x - mean_g) inv_g with
// inv_g = 1 / sqrt(var_g + eps), z = xhat gamma_c + beta_c, Y = max(z, 0)
// (relu) or z:
//   gz = dY, times [z > 0] with the ReLU (derivative taken as 0 at 0);
//   dbeta_c = sum_v gz,  dgamma_c = sum_v gz xhat,  dxhat = gz gamma_c;
//   dX = inv_g (dxhat - mean_g(dxhat) - xhat mean_g(dxhat xhat)),
// the last line from differentiating mean_g and var_g through xhat.
// dgamma / dbeta may be null.
int orc_groupnorm_backward(const double* X, int64_t n, int C, int groups, const double* gamma,
                           const double* beta, double eps, int relu, const double* dY, double* dX,
                           double* dgamma, double* dbeta) {
  if (n < 0 || C <= 0 || groups <= 0 || C % groups != 0 || !(eps >= 0.0)) return EINVAL_;
  if (n > 0 && (!X || !dY || !dX)) return EINVAL_;
  const int per = C / groups;
  if (dgamma) std::fill(dgamma, dgamma + C, 0.0);
  if (dbeta) std::fill(dbeta, dbeta + C, 0.0);
  std::vector<double> xh(static_cast<size_t>(n) * per), gz(static_cast<size_t>(n) * per);
  for (int g = 0; g < groups; ++g) {
    const double cnt = static_cast<double>(n) * per;
    if (cnt == 0) continue;
    double mean = 0.0;
    for (int64_t v = 0; v < n; ++v)
      for (int c = g * per; c < (g + 1) * per; ++c) mean += X[v * C + c];
    mean /= cnt;
    double var = 0.0;
    for (int64_t v = 0; v < n; ++v)
      for (int c = g * per; c < (g + 1) * per; ++c) var += (X[v * C + c] - mean) * (X[v * C + c] - mean);
    var /= cnt;
    const double inv = 1.0 / std::sqrt(var + eps);
    double m1 = 0.0, m2 = 0.0;   // sums of dxhat and dxhat * xhat over the group
    for (int64_t v = 0; v < n; ++v)
      for (int j = 0; j < per; ++j) {
        const int c = g * per + j;
        const double gm = gamma ? gamma[c] : 1.0;
        const double x_hat = (X[v * C + c] - mean) * inv;
        const double z = x_hat * gm + (beta ? beta[c] : 0.0);
        const double d = relu && !(z > 0.0) ? 0.0 : dY[v * C + c];
        xh[v * per + j] = x_hat;
        gz[v * per + j] = d;
        if (dbeta) dbeta[c] += d;
        if (dgamma) dgamma[c] += d * x_hat;
        m1 += d * gm;
        m2 += d * gm * x_hat;
      }
    m1 /= cnt;
    m2 /= cnt;
    for (int64_t v = 0; v < n; ++v)
      for (int j = 0; j < per; ++j) {
        const int c = g * per + j;
        const double dxh = gz[v * per + j] * (gamma ? gamma[c] : 1.0);
        dX[v * C + c] = inv * (dxh - m1 - xh[v * per + j] * m2);
      }
  }
  return OK;
}

// Backward of orc_deform_slice_classify for dL/dlogits = dZ (m x K): with f_p
// the DeformSlice output of point p,
//   dWc[j][c] = sum_p dZ[p][j] f_p[c],  dbc[j] = sum_p dZ[p][j],
//   df_p = sum_j dZ[p][j] Wc[j]   (what reaches the DeformSlice output),
// and the DeformSlice backward of df gives dX, dwv and dbeta.
// dWc / dbc may be null.
int orc_deform_slice_classify_backward(const orc_lattice* L, const double* X, int C, const double* wv,
                                       double beta, const double* Wc, int K, const double* dZ, double* dX,
                                       double* dwv, double* dbeta, double* dWc, double* dbc) {
  if (!L || !X || !wv || !Wc || C <= 0 || K <= 0 || !dX || !dwv || !dbeta || (L->m > 0 && !dZ)) return EINVAL_;
  std::vector<double> f(static_cast<size_t>(L->m) * C), df(static_cast<size_t>(L->m) * C, 0.0);
  orc_deform_slice_raw(X, C, C, L->idx.data(), L->bary.data(), L->m, wv, beta, nullptr, f.data(), nullptr);
  if (dWc) std::fill(dWc, dWc + static_cast<int64_t>(K) * C, 0.0);
  if (dbc) std::fill(dbc, dbc + K, 0.0);
  for (int64_t p = 0; p < L->m; ++p)
    for (int j = 0; j < K; ++j) {
      const double z = dZ[p * K + j];
      if (dbc) dbc[j] += z;
      for (int c = 0; c < C; ++c) {
        if (dWc) dWc[static_cast<int64_t>(j) * C + c] += z * f[p * C + c];
        df[p * C + c] += z * Wc[static_cast<int64_t>(j) * C + c];
      }
    }
  return orc_deform_slice_backward(L, X, C, wv, beta, df.data(), dX, dwv, dbeta);
}

// Distribute + PointNet backward: the gradient of orc_distribute_pointnet
// for dL/dX = dX (n x C3) with respect to the features F, the three layers'
// weights and biases, and the three normalisations' gamma and beta (same
// concatenated layout as the forward's); the positions are inputs, not
// parameters.  The maximum over J_v passes dX[v][c] to the row of J_v
// holding channel c's maximum (the first such row in J_v's order, points in
// increasing order).  Each [GN, ReLU, 1x1] block then goes backward:
//   dW_i = sum_rows dh_i a_{i-1}^T,  db_i = sum_rows dh_i,  da_{i-1} = W_i^T dh_i,
//   dh_{i-1} = the GroupNorm + ReLU backward of da_{i-1} (orc_groupnorm_backward),
// and dF_p = sum over the rows of point p (one per vertex of its simplex) of
// the feature part of dh_0.  margin (optional, n x C3): per vertex and
// channel, the largest row minus the second largest (+inf for a single
// row); where it is tiny either row is a valid choice for the maximum.
// Any output pointer may be null.
int orc_distribute_pointnet_backward(const orc_lattice* L, const double* G, const double* F, int cf,
                                     const double* gamma, const double* beta, double eps, const double* W1,
                                     const double* b1, int c1, const double* W2, const double* b2, int c2,
                                     const double* W3, const double* b3, int c3, const double* dX, double* dF,
                                     double* dW1, double* db1, double* dW2, double* db2, double* dW3, double* db3,
                                     double* dgamma, double* dbeta, double* margin) {
  if (!L || !dX || cf < 0 || c1 <= 0 || c2 <= 0 || c3 <= 0 || !W1 || !W2 || !W3 || !(eps >= 0.0)) return EINVAL_;
  if (L->m > 0 && (!G || (cf > 0 && !F))) return EINVAL_;
  const int cin = kDim + cf;
  const int widths[3] = {cin, c1, c2};
  const int outs[3] = {c1, c2, c3};
  for (int w : widths)
    if (w > 32 && w % 32 != 0) return EUNSUPPORTED;
  const int64_t n = static_cast<int64_t>(L->keys.size());
  std::vector<std::vector<int64_t>> J(n);
  for (int64_t p = 0; p < L->m; ++p)
    for (int k = 0; k < kD1; ++k) J[L->idx[p * kD1 + k]].push_back(p);
  // the distributed rows, vertex by vertex, as in the forward
  const int64_t rows = L->m * kD1;
  std::vector<int64_t> row_point, first_row(n + 1, 0);
  row_point.reserve(rows);
  std::vector<std::vector<double>> h(4), a(3);
  h[0].assign(static_cast<size_t>(rows) * cin, 0.0);
  int64_t r = 0;
  for (int64_t v = 0; v < n; ++v) {
    first_row[v] = r;
    double mu[kDim] = {0.0, 0.0, 0.0};
    for (int64_t p : J[v])
      for (int j = 0; j < kDim; ++j) mu[j] += G[p * kDim + j] / L->scale[j];
    for (int j = 0; j < kDim; ++j) mu[j] /= static_cast<double>(J[v].size());
    for (int64_t p : J[v]) {
      for (int j = 0; j < kDim; ++j) h[0][r * cin + j] = G[p * kDim + j] / L->scale[j] - mu[j];
      for (int c = 0; c < cf; ++c) h[0][r * cin + kDim + c] = F[p * cf + c];
      row_point.push_back(p);
      ++r;
    }
  }
  first_row[n] = r;
  const double* Ws[3] = {W1, W2, W3};
  const double* bs[3] = {b1, b2, b3};
  double* dWs[3] = {dW1, dW2, dW3};
  double* dbs[3] = {db1, db2, db3};
  int offs[3] = {0, cin, cin + c1};
  // forward, keeping every layer's input h and its activation a
  for (int layer = 0; layer < 3; ++layer) {
    const int ci = widths[layer], co = outs[layer];
    a[layer].assign(static_cast<size_t>(rows) * ci, 0.0);
    if (rows > 0) {
      const int st = orc_groupnorm(h[layer].data(), rows, ci, ci, ci <= 32 ? ci : 32,
                                   gamma ? gamma + offs[layer] : nullptr, beta ? beta + offs[layer] : nullptr, eps,
                                   1, a[layer].data(), ci);
      if (st != OK) return st;
    }
    h[layer + 1].assign(static_cast<size_t>(rows) * co, 0.0);
    for (int64_t q = 0; q < rows; ++q)
      for (int o = 0; o < co; ++o) {
        double acc = bs[layer] ? bs[layer][o] : 0.0;
        for (int i = 0; i < ci; ++i) acc += Ws[layer][o * ci + i] * a[layer][q * ci + i];
        h[layer + 1][q * co + o] = acc;
      }
  }
  // MaxPool backward
  std::vector<double> g(static_cast<size_t>(rows) * c3, 0.0);
  for (int64_t v = 0; v < n; ++v)
    for (int c = 0; c < c3; ++c) {
      int64_t best = -1;
      double top = -INFINITY, second = -INFINITY;
      for (int64_t q = first_row[v]; q < first_row[v + 1]; ++q) {
        const double val = h[3][q * c3 + c];
        if (best < 0 || val > top) {
          second = top;
          top = val;
          best = q;
        } else if (val > second) {
          second = val;
        }
      }
      if (best >= 0) g[best * c3 + c] = dX[v * c3 + c];
      if (margin) margin[v * c3 + c] = best >= 0 && first_row[v + 1] - first_row[v] > 1 ? top - second : INFINITY;
    }
  // the three blocks backward
  if (dgamma) std::fill(dgamma, dgamma + cin + c1 + c2, 0.0);
  if (dbeta) std::fill(dbeta, dbeta + cin + c1 + c2, 0.0);
  for (int layer = 2; layer >= 0; --layer) {
    const int ci = widths[layer], co = outs[layer];
    if (dWs[layer]) {
      std::fill(dWs[layer], dWs[layer] + static_cast<int64_t>(co) * ci, 0.0);
      for (int64_t q = 0; q < rows; ++q)
        for (int o = 0; o < co; ++o)
          for (int i = 0; i < ci; ++i) dWs[layer][o * ci + i] += g[q * co + o] * a[layer][q * ci + i];
    }
    if (dbs[layer]) {
      std::fill(dbs[layer], dbs[layer] + co, 0.0);
      for (int64_t q = 0; q < rows; ++q)
        for (int o = 0; o < co; ++o) dbs[layer][o] += g[q * co + o];
    }
    std::vector<double> da(static_cast<size_t>(rows) * ci, 0.0), dh(static_cast<size_t>(rows) * ci, 0.0);
    for (int64_t q = 0; q < rows; ++q)
      for (int i = 0; i < ci; ++i) {
        double acc = 0.0;
        for (int o = 0; o < co; ++o) acc += Ws[layer][o * ci + i] * g[q * co + o];
        da[q * ci + i] = acc;
      }
    if (rows > 0) {
      const int st = orc_groupnorm_backward(h[layer].data(), rows, ci, ci <= 32 ? ci : 32,
                                            gamma ? gamma + offs[layer] : nullptr,
                                            beta ? beta + offs[layer] : nullptr, eps, 1, da.data(), dh.data(),
                                            dgamma ? dgamma + offs[layer] : nullptr,
                                            dbeta ? dbeta + offs[layer] : nullptr);
      if (st != OK) return st;
    }
    g.swap(dh);
  }
  if (dF && cf > 0) {
    std::fill(dF, dF + L->m * cf, 0.0);
    for (int64_t q = 0; q < rows; ++q)
      for (int c = 0; c < cf; ++c) dF[row_point[q] * cf + c] += g[q * cin + kDim + c];
  }
  return OK;
}

// Round to the nearest bfloat16 (8 significant bits), ties to even, in place.
// Used where the bf16 pipeline stores activations; normal range only.
void orc_round_bf16(double* x, int64_t n) {
  for (int64_t e = 0; e < n; ++e) {
    if (x[e] == 0.0 || !std::isfinite(x[e])) continue;
    int ex = 0;
    const double f = std::frexp(x[e], &ex);            // x = f * 2^ex, 0.5 <= |f| < 1
    x[e] = std::ldexp(std::nearbyint(std::ldexp(f, 8)), ex - 8);
  }
}

}  // extern "C"

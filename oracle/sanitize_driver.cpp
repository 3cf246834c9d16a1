// Exercises every entry point of the CPU oracle on small inputs, for a build
// of the oracle with AddressSanitizer and UndefinedBehaviorSanitizer (host
// code only; test infrastructure).  Exits non-zero if a call fails; the
// sanitizers abort on any memory or undefined-behaviour error.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

extern "C" {
typedef struct Lattice orc_lattice;
void orc_axis_factors(const float* sigma, float* a);
int orc_elevate(const float* pos, int64_t m, const float* sigma, float* y);
int orc_simplex(const float* y, int64_t m, int32_t* keys, float* w);
int orc_create(const float* pos, int64_t m, int d, const float* sigma, orc_lattice** out);
int orc_coarsen(const orc_lattice* fine, orc_lattice** out);
void orc_destroy(orc_lattice* L);
int64_t orc_num_vertices(const orc_lattice* L);
int64_t orc_num_points(const orc_lattice* L);
int orc_level(const orc_lattice* L);
void orc_export_elevated(const orc_lattice* L, float* y);
void orc_export_keys(const orc_lattice* L, int32_t* keys);
void orc_export_simplices(const orc_lattice* L, int64_t* idx, float* w);
void orc_export_neighbors(const orc_lattice* L, int64_t* nbr);
void orc_export_down_table(const orc_lattice* coarse, int64_t* nbr);
void orc_export_up_table(const orc_lattice* coarse, int64_t* nbr);
int orc_splat(const orc_lattice* L, const double* F, int C, int normalize, double* X, double* wsum);
int orc_conv(const orc_lattice* dst, const orc_lattice* src, const double* X, int64_t ldx, int cin, const double* W,
             const double* bias, int cout, int relu, const int64_t* rows, int64_t nrows, double* Y, int64_t ldy);
int orc_refine(const orc_lattice* fine, const orc_lattice* coarse, const double* X, int64_t ldx, int cin,
               const double* W, const double* bias, int cout, int relu, const int64_t* rows, int64_t nrows,
               double* Y, int64_t ldy);
int orc_slice(const orc_lattice* L, const double* X, int64_t ldx, int C, const int64_t* pts, int64_t npts,
              double* out);
int orc_deform_slice(const orc_lattice* L, const double* X, int64_t ldx, int C, const double* wv, double beta,
                     const int64_t* pts, int64_t npts, double* out, double* delta);
int orc_deform_slice_classify(const orc_lattice* L, const double* X, int64_t ldx, int C, const double* wv,
                              double beta, const double* Wc, const double* bc, int K, double* logits);
int orc_groupnorm(const double* X, int64_t n, int C, int64_t ldx, int groups, const double* gamma,
                  const double* beta, double eps, int relu, double* Y, int64_t ldy);
int orc_distribute_pointnet(const orc_lattice* L, const double* G, const double* F, int cf, const double* gamma,
                            const double* beta, double eps, const double* W1, const double* b1, int c1,
                            const double* W2, const double* b2, int c2, const double* W3, const double* b3, int c3,
                            double* X);
int orc_splat_backward(const orc_lattice* L, const double* dX, int C, int normalize, double* dF);
int orc_slice_backward(const orc_lattice* L, const double* dOut, int C, double* dX);
int orc_conv_backward(const orc_lattice* dst, const orc_lattice* src, const double* X, int cin, const double* W,
                      int cout, int relu, const double* Y, const double* dY, double* dX, double* dW, double* dbias);
int orc_deform_slice_backward(const orc_lattice* L, const double* X, int C, const double* wv, double beta,
                              const double* dOut, double* dX, double* dwv, double* dbeta);
int orc_groupnorm_backward(const double* X, int64_t n, int C, int groups, const double* gamma,
                           const double* beta, double eps, int relu, const double* dY, double* dX,
                           double* dgamma, double* dbeta);
int orc_deform_slice_classify_backward(const orc_lattice* L, const double* X, int C, const double* wv,
                                       double beta, const double* Wc, int K, const double* dZ, double* dX,
                                       double* dwv, double* dbeta, double* dWc, double* dbc);
int orc_distribute_pointnet_backward(const orc_lattice* L, const double* G, const double* F, int cf,
                                     const double* gamma, const double* beta, double eps, const double* W1,
                                     const double* b1, int c1, const double* W2, const double* b2, int c2,
                                     const double* W3, const double* b3, int c3, const double* dX, double* dF,
                                     double* dW1, double* db1, double* dW2, double* db2, double* dW3, double* db3,
                                     double* dgamma, double* dbeta, double* margin);
void orc_round_bf16(double* x, int64_t n);
}

namespace {
uint64_t state = 0x9e3779b97f4a7c15ull;
double rnd() {   // splitmix64, uniform in [0, 1)
  uint64_t z = (state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return static_cast<double>(z >> 11) * 0x1.0p-53;
}
std::vector<double> vec(size_t n) {
  std::vector<double> v(n);
  for (auto& x : v) x = 2.0 * rnd() - 1.0;
  return v;
}
int failures = 0;
void need(int st, const char* what) {
  if (st != 0) {
    std::printf("FAIL %s: %d\n", what, st);
    ++failures;
  }
}
}  // namespace

int main() {
  const int64_t m = 300;
  const int C = 8, Co = 12, K = 5;
  std::vector<float> pos(3 * m), sigma = {0.15f, 0.15f, 0.15f};
  for (auto& p : pos) p = static_cast<float>(rnd());
  float a[3];
  orc_axis_factors(sigma.data(), a);
  std::vector<float> y(4 * m), w(4 * m);
  std::vector<int32_t> keys(16 * m);
  need(orc_elevate(pos.data(), m, sigma.data(), y.data()), "elevate");
  need(orc_simplex(y.data(), m, keys.data(), w.data()), "simplex");
  orc_lattice *L0 = nullptr, *L1 = nullptr, *L2 = nullptr, *E = nullptr;
  need(orc_create(pos.data(), m, 3, sigma.data(), &L0), "create");
  need(orc_coarsen(L0, &L1), "coarsen 1");
  need(orc_coarsen(L1, &L2), "coarsen 2");
  need(orc_create(pos.data(), 0, 3, sigma.data(), &E), "create empty");
  const int64_t n0 = orc_num_vertices(L0), n1 = orc_num_vertices(L1);
  if (orc_num_points(L0) != m || orc_level(L2) != 2) ++failures;
  std::vector<float> ye(4 * m), we(4 * m);
  std::vector<int32_t> ke(4 * n0);
  std::vector<int64_t> idx(4 * m), nb(9 * n0), dn(9 * n1), up(9 * n0);
  orc_export_elevated(L0, ye.data());
  orc_export_keys(L0, ke.data());
  orc_export_simplices(L0, idx.data(), we.data());
  orc_export_neighbors(L0, nb.data());
  orc_export_down_table(L1, dn.data());
  orc_export_up_table(L1, up.data());
  // forward operators
  auto F = vec(m * C), W = vec(9 * C * Co), W2 = vec(9 * Co * C), bias = vec(Co);
  std::vector<double> X(n0 * C), ws(n0), Y(n0 * Co), Y1(n1 * Co), Yr(n0 * C), out(m * C), delta(4 * m);
  need(orc_splat(L0, F.data(), C, 1, X.data(), ws.data()), "splat");
  need(orc_conv(L0, L0, X.data(), C, C, W.data(), bias.data(), Co, 1, nullptr, 0, Y.data(), Co), "conv");
  const int64_t rows[3] = {0, n0 / 2, n0 - 1};
  need(orc_conv(L0, L0, X.data(), C, C, W.data(), nullptr, Co, 0, rows, 3, Y.data(), Co), "conv rows");
  need(orc_conv(L1, L0, X.data(), C, C, W.data(), nullptr, Co, 0, nullptr, 0, Y1.data(), Co), "strided conv");
  need(orc_refine(L0, L1, Y1.data(), Co, Co, W2.data(), nullptr, C, 0, nullptr, 0, Yr.data(), C), "refine");
  need(orc_slice(L0, X.data(), C, C, nullptr, 0, out.data()), "slice");
  auto wv = vec(C);
  need(orc_deform_slice(L0, X.data(), C, C, wv.data(), 0.1, nullptr, 0, out.data(), delta.data()), "deform");
  const int64_t pts[2] = {0, m - 1};
  need(orc_deform_slice(L0, X.data(), C, C, wv.data(), 0.1, pts, 2, out.data(), delta.data()), "deform pts");
  auto Wc = vec(K * C), bc = vec(K);
  std::vector<double> logits(m * K);
  need(orc_deform_slice_classify(L0, X.data(), C, C, wv.data(), 0.1, Wc.data(), bc.data(), K, logits.data()),
       "classify");
  std::vector<double> G(n0 * C);
  need(orc_groupnorm(X.data(), n0, C, C, 4, nullptr, nullptr, 1e-5, 1, G.data(), C), "groupnorm");
  std::vector<double> Gp(3 * m);
  for (int64_t e = 0; e < 3 * m; ++e) Gp[e] = pos[e];
  const int cf = 2;
  auto Fd = vec(m * cf), P1 = vec(16 * (3 + cf)), p1 = vec(16), P2 = vec(32 * 16), p2 = vec(32), P3 = vec(16 * 32),
       p3 = vec(16), gam = vec(3 + cf + 16 + 32), bet = vec(3 + cf + 16 + 32);
  std::vector<double> D(n0 * 16);
  need(orc_distribute_pointnet(L0, Gp.data(), Fd.data(), cf, gam.data(), bet.data(), 1e-5, P1.data(), p1.data(),
                               16, P2.data(), p2.data(), 32, P3.data(), p3.data(), 16, D.data()),
       "distribute");
  // backward operators
  auto dX = vec(n0 * C), dOut = vec(m * C), dY = vec(n0 * Co);
  std::vector<double> dF(m * C), dXs(n0 * C), dXc(n0 * C), dWc(9 * C * Co), dbc(Co), dwv(C);
  double dbeta = 0.0;
  need(orc_splat_backward(L0, dX.data(), C, 1, dF.data()), "splat backward");
  need(orc_slice_backward(L0, dOut.data(), C, dXs.data()), "slice backward");
  need(orc_conv_backward(L0, L0, X.data(), C, W.data(), Co, 1, Y.data(), dY.data(), dXc.data(), dWc.data(),
                         dbc.data()),
       "conv backward");
  std::vector<double> dX1(n1 * Co), dW2(9 * Co * C), db2(C);
  need(orc_conv_backward(L0, L1, Y1.data(), Co, W2.data(), C, 0, nullptr, X.data(), dX1.data(), dW2.data(),
                         db2.data()),
       "upsample backward");
  need(orc_conv_backward(L1, L0, X.data(), C, W.data(), Co, 0, nullptr, Y1.data(), nullptr, nullptr, dbc.data()),
       "strided backward, bias only");
  need(orc_deform_slice_backward(L0, X.data(), C, wv.data(), 0.1, dOut.data(), dXs.data(), dwv.data(), &dbeta),
       "deform backward");
  auto gg = vec(C), gb = vec(C);
  std::vector<double> dXg(n0 * C), dgg(C), dgb(C);
  need(orc_groupnorm_backward(X.data(), n0, C, 4, gg.data(), gb.data(), 1e-5, 1, dX.data(), dXg.data(), dgg.data(),
                              dgb.data()),
       "groupnorm backward");
  auto dZ = vec(m * K);
  std::vector<double> dWk(K * C), dbk(K);
  need(orc_deform_slice_classify_backward(L0, X.data(), C, wv.data(), 0.1, Wc.data(), K, dZ.data(), dXs.data(),
                                          dwv.data(), &dbeta, dWk.data(), dbk.data()),
       "classify backward");
  auto dD = vec(n0 * 16);
  std::vector<double> dFd(m * cf), dP1(16 * (3 + cf)), dp1(16), dP2(32 * 16), dp2(32), dP3(16 * 32), dp3(16),
      dgam(3 + cf + 16 + 32), dbet(3 + cf + 16 + 32), marg(n0 * 16);
  need(orc_distribute_pointnet_backward(L0, Gp.data(), Fd.data(), cf, gam.data(), bet.data(), 1e-5, P1.data(),
                                        p1.data(), 16, P2.data(), p2.data(), 32, P3.data(), p3.data(), 16, dD.data(),
                                        dFd.data(), dP1.data(), dp1.data(), dP2.data(), dp2.data(), dP3.data(),
                                        dp3.data(), dgam.data(), dbet.data(), marg.data()),
       "distribute backward");
  orc_round_bf16(X.data(), n0 * C);
  orc_destroy(E);
  orc_destroy(L2);
  orc_destroy(L1);
  orc_destroy(L0);
  std::printf("%s: n0=%lld n1=%lld\n", failures ? "FAILED" : "sanitized oracle ok", static_cast<long long>(n0),
              static_cast<long long>(n1));
  return failures ? 1 : 0;
}

// Group Normalization statistics for the pre-activated convolutions
// (Implementation: every convolution is pre-activated by Group Normalization
// with 32 groups and a ReLU).  Over the n vertices of a lattice and the
// channels of each group: mean and biased variance, summed in fp64 in a fixed
// order (per-workgroup partials, then a tree over the partials).  The
// result is the per-channel affine map the convolution applies to every
// gathered input value before its ReLU:
//   scale_c = gamma_c / sqrt(var_g + eps),  shift_c = beta_c - mean_g scale_c.
#include <algorithm>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int kGnMaxParts = 2048;
constexpr int kGnMinRows = 128;

// Workgroup w sums rows [w * rows_per, (w + 1) * rows_per): thread t takes
// the EPT channels EPT (t % groups_of_c) .. + EPT - 1 (16 bytes: 8 bf16 or 4
// fp32) of rows t / groups_of_c, + slots, ...; the slots are then added in
// order.
template <bool BF16>
__global__ void __launch_bounds__(kBlock)
k_gn_partial(const void* __restrict__ x, int64_t ld, int C, int64_t n, int64_t rows_per,
             double* __restrict__ part) {
  constexpr int EPT = BF16 ? 8 : 4;
  __shared__ double sh[2][kBlock][EPT];
  const int t = threadIdx.x;
  const int quads = C / EPT;
  const int slots = kBlock / quads;
  const int q = t % quads, slot = t / quads;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rows_per;
  const int64_t r1 = min(r0 + rows_per, n);
  double s[EPT], ss[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i) s[i] = ss[i] = 0.0;
  if (slot < slots) {
    for (int64_t v = r0 + slot; v < r1; v += slots) {
      float f[EPT];
      if constexpr (BF16) {
        const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + v * ld + EPT * q);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f[2 * i] = __uint_as_float(w[i] << 16);
          f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
      } else {
        const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + v * ld + EPT * q);
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
      }
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        s[i] += f[i];
        ss[i] += static_cast<double>(f[i]) * f[i];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    sh[0][t][i] = s[i];
    sh[1][t][i] = ss[i];
  }
  __syncthreads();
  // thread q < quads: its EPT channels summed over the slots in order
  if (t < quads) {
    double a[EPT], b[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) a[i] = b[i] = 0.0;
    for (int sl = 0; sl < slots; ++sl)
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        a[i] += sh[0][sl * quads + t][i];
        b[i] += sh[1][sl * quads + t][i];
      }
    double* p = part + static_cast<int64_t>(blockIdx.x) * 2 * C;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      p[EPT * t + i] = a[i];
      p[C + EPT * t + i] = b[i];
    }
  }
}

// One workgroup per group: the threads stride over the partials (and the
// group's channels), then a fixed tree adds their sums; writes scale
// (pre[0..C)) and shift (pre[C..2C)) of the group's channels, and when
// stats is given the group's mean and 1 / sqrt(var + eps).
__global__ void __launch_bounds__(kBlock)
k_gn_finalize(const double* __restrict__ part, int nparts, int C, int groups, int64_t n,
              const float* __restrict__ gamma, const float* __restrict__ beta, float eps, float* __restrict__ pre,
              double* __restrict__ stats) {
  __shared__ double sh[2][kBlock];
  const int g = blockIdx.x;
  const int per = C / groups;
  const int t = threadIdx.x;
  double s = 0.0, ss = 0.0;
  // unrolled so that the loads of several partials are in flight at once;
  // they are still added in q order
#pragma unroll 8
  for (int64_t q = t; q < static_cast<int64_t>(nparts) * per; q += kBlock) {
    const int64_t w = q / per;
    const int c = g * per + static_cast<int>(q - w * per);
    s += part[w * 2 * C + c];
    ss += part[w * 2 * C + C + c];
  }
  sh[0][t] = s;
  sh[1][t] = ss;
  __syncthreads();
  for (int off = kBlock / 2; off > 0; off >>= 1) {
    if (t < off) {
      sh[0][t] += sh[0][t + off];
      sh[1][t] += sh[1][t + off];
    }
    __syncthreads();
  }
  const double cnt = static_cast<double>(n) * per;
  const double mean = cnt > 0 ? sh[0][0] / cnt : 0.0;
  const double var = cnt > 0 ? max(sh[1][0] / cnt - mean * mean, 0.0) : 0.0;
  const double inv = 1.0 / sqrt(var + static_cast<double>(eps));
  if (stats && t == 0) {
    stats[2 * g] = mean;
    stats[2 * g + 1] = inv;
  }
  for (int c = g * per + t; c < (g + 1) * per; c += kBlock) {
    const double sc = (gamma ? gamma[c] : 1.0) * inv;
    pre[c] = static_cast<float>(sc);
    pre[C + c] = static_cast<float>((beta ? beta[c] : 0.0) - mean * sc);
  }
}

// The pre-activated input a = max(x scale_c + shift_c, 0), computed with
// the same fused multiply-add as the convolution's gather, so that it is
// bit-identical to what the forward multiplied.
__global__ void __launch_bounds__(kBlock)
k_gn_relu_apply(const float* __restrict__ x, int64_t ldx, int C, int64_t n, const float* __restrict__ pre,
                float* __restrict__ a, int64_t lda) {
  const int quads = C / 4;
  const int64_t total = n * quads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t v = i / quads;
    const int c = 4 * static_cast<int>(i - v * quads);
    const float4 xv = *reinterpret_cast<const float4*>(x + v * ldx + c);
    const float4 sc = *reinterpret_cast<const float4*>(pre + c);
    const float4 sh = *reinterpret_cast<const float4*>(pre + C + c);
    *reinterpret_cast<float4*>(a + v * lda + c) =
        make_float4(fmaxf(fmaf(xv.x, sc.x, sh.x), 0.f), fmaxf(fmaf(xv.y, sc.y, sh.y), 0.f),
                    fmaxf(fmaf(xv.z, sc.z, sh.z), 0.f), fmaxf(fmaf(xv.w, sc.w, sh.w), 0.f));
  }
}

// Backward of GroupNorm + ReLU, first pass: per-channel sums over the rows
// of workgroup w's range (fp64, rows in the order of k_gn_partial)
//   S1_c = sum g,  S2_c = sum g xhat,
// g = dA where the ReLU passed (else 0), xhat = (x - mean_g) inv_g (x itself
// when the rows given are already normalised); the ReLU passed where act > 0
// when the activations act are given, else where x scale_c + shift_c > 0.
// part[w][0..C) holds S1, part[w][C..2C) S2.
__global__ void __launch_bounds__(kBlock)
k_gn_bwd_partial(const float* __restrict__ x, int64_t ldx, const float* __restrict__ dA, int64_t lda, int C,
                 int groups, int64_t n, int64_t rows_per, const float* __restrict__ pre,
                 const float* __restrict__ act, int64_t ldact, const double* __restrict__ stats, int xhat,
                 double* __restrict__ part) {
  __shared__ double sh[2][kBlock][4];
  const int t = threadIdx.x;
  const int quads = C / 4;
  const int slots = kBlock / quads;
  const int q = t % quads, slot = t / quads;
  const int per = C / groups;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rows_per;
  const int64_t r1 = min(r0 + rows_per, n);
  double s[4] = {0.0, 0.0, 0.0, 0.0}, ss[4] = {0.0, 0.0, 0.0, 0.0};
  if (slot < slots) {
    float sc[4], sf[4];
    double mu[4], iv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 4 * q + i;
      sc[i] = pre ? pre[c] : 0.f;
      sf[i] = pre ? pre[C + c] : 0.f;
      mu[i] = xhat ? 0.0 : stats[2 * (c / per)];
      iv[i] = xhat ? 1.0 : stats[2 * (c / per) + 1];
    }
    for (int64_t v = r0 + slot; v < r1; v += slots) {
      const float4 a = *reinterpret_cast<const float4*>(x + v * ldx + 4 * q);
      const float4 d = *reinterpret_cast<const float4*>(dA + v * lda + 4 * q);
      const float xv[4] = {a.x, a.y, a.z, a.w}, dv[4] = {d.x, d.y, d.z, d.w};
      bool on[4];
      if (act) {
        const float4 u = *reinterpret_cast<const float4*>(act + v * ldact + 4 * q);
        on[0] = u.x > 0.f; on[1] = u.y > 0.f; on[2] = u.z > 0.f; on[3] = u.w > 0.f;
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) on[i] = fmaf(xv[i], sc[i], sf[i]) > 0.f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double g = on[i] ? static_cast<double>(dv[i]) : 0.0;
        s[i] += g;
        ss[i] += g * ((static_cast<double>(xv[i]) - mu[i]) * iv[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sh[0][t][i] = s[i];
    sh[1][t][i] = ss[i];
  }
  __syncthreads();
  if (t < quads) {
    double a[4] = {0.0, 0.0, 0.0, 0.0}, b[4] = {0.0, 0.0, 0.0, 0.0};
    for (int sl = 0; sl < slots; ++sl)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] += sh[0][sl * quads + t][i];
        b[i] += sh[1][sl * quads + t][i];
      }
    double* p = part + static_cast<int64_t>(blockIdx.x) * 2 * C;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[4 * t + i] = a[i];
      p[C + 4 * t + i] = b[i];
    }
  }
}

// Second pass, one workgroup per group: the channels' totals over the
// partials (each summed in a fixed order), dbeta_c = S1_c, dgamma_c = S2_c,
// and the coefficients of the input gradient of every channel c of the group
//   dX = g c1 + c0 + (x - mean) cx,
//   c1 = inv gamma_c,  c0 = -inv A,  cx = -inv^2 B,
//   A = sum_c gamma_c S1_c / N,  B = sum_c gamma_c S2_c / N  (N = n per),
// stored as coef[c] = (c1, c0, cx, mean); for rows given normalised,
// dX = g c1 + c0 + xhat (-inv B), stored as (c1, c0, -inv B, 0).
__global__ void __launch_bounds__(kBlock)
k_gn_bwd_finalize(const double* __restrict__ part, int nparts, int C, int groups, int64_t n,
                  const float* __restrict__ gamma, const double* __restrict__ stats, int xhat,
                  float* __restrict__ dgamma, float* __restrict__ dbeta, float4* __restrict__ coef) {
  __shared__ double sh[2][kBlock];
  __shared__ double tot[2][kBlock];
  __shared__ double ab[2];
  const int g = blockIdx.x;
  const int per = C / groups;
  const int t = threadIdx.x;
  double A = 0.0, B = 0.0;   // thread 0: the group's sums, channels in order
  for (int cb = 0; cb < per; cb += kBlock) {
    const int wdt = min(per - cb, kBlock);
    const int slices = kBlock / wdt;
    const int j = t % wdt, k = t / wdt;
    const int c = g * per + cb + j;
    double s = 0.0, ss = 0.0;
    if (k < slices)
#pragma unroll 8
      for (int w = k; w < nparts; w += slices) {
        s += part[static_cast<int64_t>(w) * 2 * C + c];
        ss += part[static_cast<int64_t>(w) * 2 * C + C + c];
      }
    sh[0][t] = s;
    sh[1][t] = ss;
    __syncthreads();
    if (t < wdt) {
      double a = 0.0, b = 0.0;
      for (int kk = 0; kk < slices; ++kk) {
        a += sh[0][kk * wdt + t];
        b += sh[1][kk * wdt + t];
      }
      if (dbeta) dbeta[c] = static_cast<float>(a);
      if (dgamma) dgamma[c] = static_cast<float>(b);
      const double gm = gamma ? gamma[c] : 1.0;
      tot[0][t] = gm * a;
      tot[1][t] = gm * b;
    }
    __syncthreads();
    if (t == 0)
      for (int jj = 0; jj < wdt; ++jj) {
        A += tot[0][jj];
        B += tot[1][jj];
      }
    __syncthreads();
  }
  const double cnt = static_cast<double>(n) * per;
  if (t == 0) {
    ab[0] = cnt > 0 ? A / cnt : 0.0;
    ab[1] = cnt > 0 ? B / cnt : 0.0;
  }
  __syncthreads();
  if (coef) {
    const double mean = stats[2 * g], inv = stats[2 * g + 1];
    for (int c = g * per + t; c < (g + 1) * per; c += kBlock) {
      const double gm = gamma ? gamma[c] : 1.0;
      coef[c] = make_float4(static_cast<float>(inv * gm), static_cast<float>(-inv * ab[0]),
                            static_cast<float>(xhat ? -inv * ab[1] : -inv * inv * ab[1]),
                            static_cast<float>(xhat ? 0.0 : mean));
    }
  }
}

// Third pass: dX = g c1 + c0 + (x - mean) cx, with g = dA masked as above.
__global__ void __launch_bounds__(kBlock)
k_gn_bwd_apply(const float* __restrict__ x, int64_t ldx, const float* __restrict__ dA, int64_t lda, int C, int64_t n,
               const float* __restrict__ pre, const float* __restrict__ act, int64_t ldact,
               const float4* __restrict__ coef, float* __restrict__ dX, int64_t lddx) {
  const int quads = C / 4;
  const int64_t total = n * quads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t v = i / quads;
    const int c = 4 * static_cast<int>(i - v * quads);
    const float4 a = *reinterpret_cast<const float4*>(x + v * ldx + c);
    const float4 d = *reinterpret_cast<const float4*>(dA + v * lda + c);
    const float xv[4] = {a.x, a.y, a.z, a.w}, dv[4] = {d.x, d.y, d.z, d.w};
    bool on[4];
    if (act) {
      const float4 u = *reinterpret_cast<const float4*>(act + v * ldact + c);
      on[0] = u.x > 0.f; on[1] = u.y > 0.f; on[2] = u.z > 0.f; on[3] = u.w > 0.f;
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) on[k] = fmaf(xv[k], pre[c + k], pre[C + c + k]) > 0.f;
    }
    float o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float g = on[k] ? dv[k] : 0.f;
      const float4 cf = coef[c + k];
      o[k] = fmaf(xv[k] - cf.w, cf.z, fmaf(g, cf.x, cf.y));
    }
    *reinterpret_cast<float4*>(dX + v * lddx + c) = make_float4(o[0], o[1], o[2], o[3]);
  }
}

inline unsigned elementwise_grid(int64_t n, int C) {
  const int64_t b = (n * (C / 4) + kBlock - 1) / kBlock;
  return static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(b, 8192)));
}

// Rows per partial: at least kGnMinRows (small levels then leave a few
// hundred partials, which the finalize reads in one or two loads per
// thread), at most 2,048 partials on large ones.
void gn_parts(int64_t n, int C, int bf16, int64_t* nparts, int64_t* rows_per) {
  const int slots = kBlock / (C / (bf16 ? 8 : 4));
  int64_t rp = std::max<int64_t>(std::max<int64_t>(slots, kGnMinRows), (n + kGnMaxParts - 1) / kGnMaxParts);
  rp = (rp + slots - 1) / slots * slots;
  *rows_per = rp;
  *nparts = std::max<int64_t>(1, (n + rp - 1) / rp);
}

}  // namespace

void launch_gn_finalize(const double* part, int64_t nparts, int C, int groups, int64_t rows, const float* gamma,
                        const float* beta, float eps, float* pre, hipStream_t s, double* stats) {
  launch(k_gn_finalize, dim3(static_cast<unsigned>(groups)), dim3(kBlock), 0, s, part,
         rows > 0 ? static_cast<int>(nparts) : 0, C, groups, rows, gamma, beta, eps, pre, stats);
}

int gn_max_channels() { return 4 * kBlock; }

int64_t gn_workspace_bytes(int64_t n, int C) {
  int64_t np, rp;
  gn_parts(n, C, 0, &np, &rp);   // fp32 splits into at least as many parts as bf16
  return np * 2 * C * static_cast<int64_t>(sizeof(double));
}

void launch_gn_affine(const void* x, int64_t ld, int C, int bf16, int64_t n, int groups, const float* gamma,
                      const float* beta, float eps, float* pre, void* work, hipStream_t s, double* stats) {
  ScopedKernelTimer tm("groupnorm", s);
  int64_t np, rp;
  gn_parts(n, C, bf16, &np, &rp);
  double* part = static_cast<double*>(work);
  if (n > 0) {
    if (bf16) launch(k_gn_partial<true>, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, x, ld, C, n, rp, part);
    else launch(k_gn_partial<false>, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, x, ld, C, n, rp, part);
  }
  launch(k_gn_finalize, dim3(static_cast<unsigned>(groups)), dim3(kBlock), 0, s,
         static_cast<const double*>(part), n > 0 ? static_cast<int>(np) : 0, C, groups, n, gamma, beta, eps, pre,
         stats);
}

void launch_gn_relu_apply(const float* x, int64_t ldx, int C, int64_t n, const float* pre, float* a, int64_t lda,
                          hipStream_t s) {
  if (n <= 0) return;
  launch(k_gn_relu_apply, dim3(elementwise_grid(n, C)), dim3(kBlock), 0, s, x, ldx, C, n, pre, a, lda);
}

void launch_gn_backward(const float* x, int64_t ldx, const float* dA, int64_t lda, int C, int groups, int64_t n,
                        const float* gamma, const float* pre, const double* stats, float* dgamma, float* dbeta,
                        float* coef, float* dX, int64_t lddx, void* work, hipStream_t s, const float* act,
                        int64_t ldact, bool xhat) {
  ScopedKernelTimer tm("groupnorm_bwd", s);
  int64_t np, rp;
  gn_parts(n, C, 0, &np, &rp);
  double* part = static_cast<double*>(work);
  if (n > 0)
    launch(k_gn_bwd_partial, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, x, ldx, dA, lda, C, groups, n, rp,
           pre, act, ldact, stats, xhat ? 1 : 0, part);
  launch(k_gn_bwd_finalize, dim3(static_cast<unsigned>(groups)), dim3(kBlock), 0, s,
         static_cast<const double*>(part), n > 0 ? static_cast<int>(np) : 0, C, groups, n, gamma, stats, xhat ? 1 : 0,
         dgamma, dbeta, dX ? reinterpret_cast<float4*>(coef) : nullptr);
  if (dX && n > 0)
    launch(k_gn_bwd_apply, dim3(elementwise_grid(n, C)), dim3(kBlock), 0, s, x, ldx, dA, lda, C, n, pre, act, ldact,
           reinterpret_cast<const float4*>(coef), dX, lddx);
}

}  // namespace lat

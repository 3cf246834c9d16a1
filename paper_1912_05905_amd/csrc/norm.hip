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
// (pre[0..C)) and shift (pre[C..2C)) of the group's channels.
__global__ void __launch_bounds__(kBlock)
k_gn_finalize(const double* __restrict__ part, int nparts, int C, int groups, int64_t n,
              const float* __restrict__ gamma, const float* __restrict__ beta, float eps, float* __restrict__ pre) {
  __shared__ double sh[2][kBlock];
  const int g = blockIdx.x;
  const int per = C / groups;
  const int t = threadIdx.x;
  double s = 0.0, ss = 0.0;
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
  for (int c = g * per + t; c < (g + 1) * per; c += kBlock) {
    const double sc = (gamma ? gamma[c] : 1.0) * inv;
    pre[c] = static_cast<float>(sc);
    pre[C + c] = static_cast<float>((beta ? beta[c] : 0.0) - mean * sc);
  }
}

void gn_parts(int64_t n, int C, int bf16, int64_t* nparts, int64_t* rows_per) {
  const int slots = kBlock / (C / (bf16 ? 8 : 4));
  int64_t rp = std::max<int64_t>(slots, (n + kGnMaxParts - 1) / kGnMaxParts);
  rp = (rp + slots - 1) / slots * slots;
  *rows_per = rp;
  *nparts = std::max<int64_t>(1, (n + rp - 1) / rp);
}

}  // namespace

void launch_gn_finalize(const double* part, int64_t nparts, int C, int groups, int64_t rows, const float* gamma,
                        const float* beta, float eps, float* pre, hipStream_t s) {
  launch(k_gn_finalize, dim3(static_cast<unsigned>(groups)), dim3(kBlock), 0, s, part,
         rows > 0 ? static_cast<int>(nparts) : 0, C, groups, rows, gamma, beta, eps, pre);
}

int gn_max_channels() { return 4 * kBlock; }

int64_t gn_workspace_bytes(int64_t n, int C) {
  int64_t np, rp;
  gn_parts(n, C, 0, &np, &rp);   // fp32 splits into at least as many parts as bf16
  return np * 2 * C * static_cast<int64_t>(sizeof(double));
}

void launch_gn_affine(const void* x, int64_t ld, int C, int bf16, int64_t n, int groups, const float* gamma,
                      const float* beta, float eps, float* pre, void* work, hipStream_t s) {
  ScopedKernelTimer tm("groupnorm", s);
  int64_t np, rp;
  gn_parts(n, C, bf16, &np, &rp);
  double* part = static_cast<double*>(work);
  if (n > 0) {
    if (bf16) launch(k_gn_partial<true>, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, x, ld, C, n, rp, part);
    else launch(k_gn_partial<false>, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, x, ld, C, n, rp, part);
  }
  launch(k_gn_finalize, dim3(static_cast<unsigned>(groups)), dim3(kBlock), 0, s,
         static_cast<const double*>(part), n > 0 ? static_cast<int>(np) : 0, C, groups, n, gamma, beta, eps, pre);
}

}  // namespace lat

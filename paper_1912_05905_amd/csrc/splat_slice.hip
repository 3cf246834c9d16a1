// Splat, Slice and DeformSlice on gfx950.  All three are gathers bounded by
// HBM bandwidth: a row of C channels is handled by a group of LPR lanes
// (LPR a power of two), each lane moving 16 bytes (4 fp32 or 8 bf16 channels)
// per access so that a row is one contiguous, fully used transaction.
#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;

// float -> bfloat16, round to nearest even (NaN stays NaN).
__device__ inline uint16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// A 16-byte chunk of a row as 8 floats (bf16) or 4 floats (fp32).
template <bool BF16> struct Chunk;
template <> struct Chunk<false> {
  static constexpr int N = 4;
  float v[4];
  __device__ inline void load(const void* base, int64_t elem) {
    const float4 x = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  }
  __device__ inline void store(void* base, int64_t elem) const {
    *reinterpret_cast<float4*>(static_cast<float*>(base) + elem) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct Chunk<true> {
  static constexpr int N = 8;
  float v[8];
  __device__ inline void load(const void* base, int64_t elem) {
    const uint4 x = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ inline void store(void* base, int64_t elem) const {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = static_cast<uint32_t>(f32_to_bf16(v[2 * i])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * i + 1])) << 16);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(base) + elem) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Splat (Eq. splat) as a gather over J_v: one lane group per vertex reads
// the vertex's (point, weight) list and accumulates b * f in fp32.  Lane i of
// the group fetches list entry s+i; the group then walks the batch with
// shuffles, so LPR feature rows are in flight at once.  No float atomics.
template <bool BF16, int LPR>
__global__ void __launch_bounds__(kBlock)
k_splat(const int32_t* __restrict__ offsets, const int32_t* __restrict__ entries,
        const float* __restrict__ entry_w, const void* __restrict__ feat, int64_t ld_feat, int C,
        int normalize, int64_t n, void* __restrict__ vals, int64_t ld_vals, float* __restrict__ wsum) {
  using Ch = Chunk<BF16>;
  constexpr int kMaxChunks = 4;                  // up to 4*LPR chunks per row
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t v = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / LPR;
  const bool live = v < n;
  const int nchunk = C / Ch::N;
  float acc[kMaxChunks][Ch::N];
#pragma unroll
  for (int q = 0; q < kMaxChunks; ++q)
#pragma unroll
    for (int e = 0; e < Ch::N; ++e) acc[q][e] = 0.f;
  float ws = 0.f;
  const int32_t beg = live ? offsets[v] : 0;
  const int32_t end = live ? offsets[v + 1] : 0;
  for (int32_t s = beg; s < end; s += LPR) {
    const int cnt = min(LPR, end - s);
    int32_t my_e = 0;
    float my_w = 0.f;
    if (lane < cnt) {
      my_e = entries[s + lane];
      my_w = entry_w[s + lane];
    }
    for (int j = 0; j < cnt; ++j) {
      const int32_t e = __shfl(my_e, j, LPR);
      const float wt = __shfl(my_w, j, LPR);
      const int64_t p = e >> 2;
      ws += wt;
#pragma unroll
      for (int q = 0; q < kMaxChunks; ++q) {
        const int ch = lane + q * LPR;
        if (ch < nchunk) {
          Ch f;
          f.load(feat, p * ld_feat + static_cast<int64_t>(ch) * Ch::N);
#pragma unroll
          for (int i = 0; i < Ch::N; ++i) acc[q][i] += wt * f.v[i];
        }
      }
    }
  }
  if (!live) return;
  const float scale = normalize ? (ws > 0.f ? 1.0f / ws : 0.f) : 1.0f;
#pragma unroll
  for (int q = 0; q < kMaxChunks; ++q) {
    const int ch = lane + q * LPR;
    if (ch < nchunk) {
      Ch o;
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) o.v[i] = normalize ? acc[q][i] * scale : acc[q][i];
      o.store(vals, v * ld_vals + static_cast<int64_t>(ch) * Ch::N);
    }
  }
  if (wsum && lane == 0) wsum[v] = ws;
}

// Slice (Eq. slice): out_p = sum_k b_pk x_{idx_pk}; one lane group per point.
template <bool BF16, int LPR>
__global__ void __launch_bounds__(kBlock)
k_slice(const int4* __restrict__ idx, const float4* __restrict__ w, int64_t m,
        const void* __restrict__ vals, int64_t ld_vals, int C, float* __restrict__ out) {
  using Ch = Chunk<BF16>;
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t p = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / LPR;
  if (p >= m) return;
  const int4 iv = idx[p];
  const float4 wv = w[p];
  const int32_t vi[4] = {iv.x, iv.y, iv.z, iv.w};
  const float bw[4] = {wv.x, wv.y, wv.z, wv.w};
  const int nchunk = C / Ch::N;
  for (int ch = lane; ch < nchunk; ch += LPR) {
    float acc[Ch::N];
#pragma unroll
    for (int i = 0; i < Ch::N; ++i) acc[i] = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (vi[k] < 0) continue;
      Ch x;
      x.load(vals, static_cast<int64_t>(vi[k]) * ld_vals + static_cast<int64_t>(ch) * Ch::N);
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[i] += bw[k] * x.v[i];
    }
    float* o = out + p * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
    for (int i = 0; i < Ch::N; i += 4)
      *reinterpret_cast<float4*>(o + i) = make_float4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
  }
}

// DeformSlice (Eq. deformSlice): q_k = b_k x_k; M = max_k q_k per channel;
// db_k = tanh(beta + (q_k - M) . wv); out = sum_k (b_k + db_k) x_k.
// Each lane keeps its channels of the d+1 gathered rows in registers; the
// dot products are reduced across the lane group with xor shuffles.
template <bool BF16, int LPR, int CPL>
__global__ void __launch_bounds__(kBlock)
k_deform_slice(const int4* __restrict__ idx, const float4* __restrict__ w, int64_t m,
               const void* __restrict__ vals, int64_t ld_vals, int C, const float* __restrict__ wvec,
               float beta, float* __restrict__ out, float4* __restrict__ delta) {
  using Ch = Chunk<BF16>;
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t p = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / LPR;
  const bool live = p < m;
  const int nchunk = C / Ch::N;
  int4 iv = make_int4(-1, -1, -1, -1);
  float4 wq = make_float4(0.f, 0.f, 0.f, 0.f);
  if (live) { iv = idx[p]; wq = w[p]; }
  const int32_t vi[4] = {iv.x, iv.y, iv.z, iv.w};
  const float bw[4] = {wq.x, wq.y, wq.z, wq.w};
  float x[CPL][4][Ch::N];
  float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int ch = lane + q * LPR;
    const bool on = live && ch < nchunk;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (on && vi[k] >= 0) {
        Ch c;
        c.load(vals, static_cast<int64_t>(vi[k]) * ld_vals + static_cast<int64_t>(ch) * Ch::N);
#pragma unroll
        for (int i = 0; i < Ch::N; ++i) x[q][k][i] = c.v[i];
      } else {
#pragma unroll
        for (int i = 0; i < Ch::N; ++i) x[q][k][i] = 0.f;
      }
    }
    if (on) {
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) {
        const float wc = wvec[ch * Ch::N + i];
        float qk[4];
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          qk[k] = bw[k] * x[q][k][i];
          mx = fmaxf(mx, qk[k]);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) part[k] += (qk[k] - mx) * wc;
      }
    }
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) part[k] += __shfl_xor(part[k], off, LPR);
  if (!live) return;
  float coef[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float db = tanhf(beta + part[k]);
    part[k] = db;
    coef[k] = bw[k] + db;
  }
  if (delta && lane == 0) delta[p] = make_float4(part[0], part[1], part[2], part[3]);
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int ch = lane + q * LPR;
    if (ch >= nchunk) continue;
    float* o = out + p * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
    for (int i = 0; i < Ch::N; i += 4) {
      float r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        r[u] = coef[0] * x[q][0][i + u] + coef[1] * x[q][1][i + u] + coef[2] * x[q][2][i + u] +
               coef[3] * x[q][3][i + u];
      *reinterpret_cast<float4*>(o + i) = make_float4(r[0], r[1], r[2], r[3]);
    }
  }
}

// lanes per row: enough 16-byte chunks to cover C, at most 64 (a wavefront)
inline int lanes_per_row(int C, bool bf16) {
  const int chunks = C / (bf16 ? 8 : 4);
  int l = 1;
  while (l < chunks && l < 64) l <<= 1;
  return l;
}

inline unsigned grid_for(int64_t rows, int lpr) {
  return static_cast<unsigned>((rows * lpr + kBlock - 1) / kBlock);
}

template <bool BF16>
void splat_dispatch(int lpr, const int32_t* off, const int32_t* ent, const float* ew, const void* feat,
                    int64_t ldf, int C, int norm, int64_t n, void* vals, int64_t ldv, float* wsum,
                    hipStream_t s) {
  const dim3 g(grid_for(n, lpr)), b(kBlock);
  switch (lpr) {
    case 1: hipLaunchKernelGGL((k_splat<BF16, 1>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    case 2: hipLaunchKernelGGL((k_splat<BF16, 2>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    case 4: hipLaunchKernelGGL((k_splat<BF16, 4>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    case 8: hipLaunchKernelGGL((k_splat<BF16, 8>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    case 16: hipLaunchKernelGGL((k_splat<BF16, 16>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    case 32: hipLaunchKernelGGL((k_splat<BF16, 32>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
    default: hipLaunchKernelGGL((k_splat<BF16, 64>), g, b, 0, s, off, ent, ew, feat, ldf, C, norm, n, vals, ldv, wsum); break;
  }
}

template <bool BF16>
void slice_dispatch(int lpr, const int32_t* idx, const float* w, int64_t m, const void* vals,
                    int64_t ldv, int C, float* out, hipStream_t s) {
  const dim3 g(grid_for(m, lpr)), b(kBlock);
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  switch (lpr) {
    case 1: hipLaunchKernelGGL((k_slice<BF16, 1>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    case 2: hipLaunchKernelGGL((k_slice<BF16, 2>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    case 4: hipLaunchKernelGGL((k_slice<BF16, 4>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    case 8: hipLaunchKernelGGL((k_slice<BF16, 8>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    case 16: hipLaunchKernelGGL((k_slice<BF16, 16>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    case 32: hipLaunchKernelGGL((k_slice<BF16, 32>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
    default: hipLaunchKernelGGL((k_slice<BF16, 64>), g, b, 0, s, i4, w4, m, vals, ldv, C, out); break;
  }
}

template <bool BF16, int CPL>
void deform_dispatch(int lpr, const int32_t* idx, const float* w, int64_t m, const void* vals,
                     int64_t ldv, int C, const float* wv, float beta, float* out, float* delta,
                     hipStream_t s) {
  const dim3 g(grid_for(m, lpr)), b(kBlock);
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  float4* d4 = reinterpret_cast<float4*>(delta);
  switch (lpr) {
    case 1: hipLaunchKernelGGL((k_deform_slice<BF16, 1, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    case 2: hipLaunchKernelGGL((k_deform_slice<BF16, 2, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    case 4: hipLaunchKernelGGL((k_deform_slice<BF16, 4, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    case 8: hipLaunchKernelGGL((k_deform_slice<BF16, 8, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    case 16: hipLaunchKernelGGL((k_deform_slice<BF16, 16, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    case 32: hipLaunchKernelGGL((k_deform_slice<BF16, 32, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
    default: hipLaunchKernelGGL((k_deform_slice<BF16, 64, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4); break;
  }
}

}  // namespace

// Largest channel count the gather kernels handle: 4 chunks per lane of a
// full wavefront for splat, 2 for DeformSlice; slice loops without limit.
int splat_max_channels(bool bf16) { return (bf16 ? 8 : 4) * 64 * 4; }
int deform_max_channels(bool bf16) { return (bf16 ? 8 : 4) * 64 * 2; }

void launch_splat(const int32_t* offsets, const int32_t* entries, const float* entry_w, const void* feat,
                  int64_t ld_feat, int C, int bf16, int normalize, int64_t n, void* vals,
                  int64_t ld_vals, float* wsum, hipStream_t s) {
  if (n <= 0) return;
  const int lpr = lanes_per_row(C, bf16 != 0);
  ScopedKernelTimer tm("splat", s);
  if (bf16) splat_dispatch<true>(lpr, offsets, entries, entry_w, feat, ld_feat, C, normalize, n, vals, ld_vals, wsum, s);
  else splat_dispatch<false>(lpr, offsets, entries, entry_w, feat, ld_feat, C, normalize, n, vals, ld_vals, wsum, s);
}

void launch_slice(const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ld_vals,
                  int C, int bf16, float* out, hipStream_t s) {
  if (m <= 0) return;
  const int lpr = lanes_per_row(C, bf16 != 0);
  ScopedKernelTimer tm("slice", s);
  if (bf16) slice_dispatch<true>(lpr, idx, w, m, vals, ld_vals, C, out, s);
  else slice_dispatch<false>(lpr, idx, w, m, vals, ld_vals, C, out, s);
}

void launch_deform_slice(const int32_t* idx, const float* w, int64_t m, const void* vals,
                         int64_t ld_vals, int C, int bf16, const float* wv, float beta, float* out,
                         float* delta, hipStream_t s) {
  if (m <= 0) return;
  const int lpr = lanes_per_row(C, bf16 != 0);
  const int chunks = C / (bf16 ? 8 : 4);
  ScopedKernelTimer tm("deform_slice", s);
  const bool two = chunks > lpr;
  if (bf16) {
    if (two) deform_dispatch<true, 2>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, s);
    else deform_dispatch<true, 1>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, s);
  } else {
    if (two) deform_dispatch<false, 2>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, s);
    else deform_dispatch<false, 1>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, s);
  }
}

}  // namespace lat

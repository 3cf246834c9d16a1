// Backward passes of the lattice operators on gfx950 (Implementation: the
// lattice operators have forward and backward passes on the GPU).  Every
// gradient is that of its forward operator for a scalar loss with
// dL/d(output) given; the linear operators' gradients are their adjoints:
//   splat  -> a slice of dL/dx (each vertex row scaled by 1 / sum_{J_v} b
//             when the forward normalised);
//   slice  -> a (raw) splat of dL/df over the lists J_v;
//   conv   -> dX: the convolution of dL/dY with W'[t] = W[mirror t]^T over
//             the adjoint table (1-hop: the same table; strided: the
//             Upsample table; Upsample: the Downsample table), on the
//             forward's MFMA kernel;
//             dW[t] = sum_v dL/dY_v^T X[nb(v,t)], dbias = sum_v dL/dY_v: a
//             gathered GEMM that reduces over vertices (k_conv_wgrad, split
//             over vertex chunks, partials added in chunk order).
// A ReLU in the forward masks dL/dY with Y > 0 first (derivative 0 at 0).
//   classifier fused with DeformSlice -> with f_p the DeformSlice output and
//             z_p = dL/dlogits_p: df_p = sum_j z_pj Wc[j] (then the
//             DeformSlice backward), dWc = sum_p z_p f_p^T, dbc = sum_p z_p
//             (point chunks, partials added in chunk order).
#include <algorithm>
#include <type_traits>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---- splat backward with normalisation: rows of dL/dx divided by the
// vertex weight sums ----
// One group of 16 lanes per vertex: the weight sum comes from the forward
// (wsum) or is summed over J_v by the lanes; the vertex's row is then
// scaled (0 where the sum is 0, as in the forward).
constexpr int kScaleLanes = 16;

__global__ void __launch_bounds__(kBlock)
k_scale_by_weight_sum(const int32_t* __restrict__ offsets, const float* __restrict__ entry_w,
                      const float* __restrict__ wsum, int64_t n, const float* __restrict__ in, int64_t ld_in, int C,
                      float* __restrict__ out, int64_t ld_out) {
  const int lane = threadIdx.x & (kScaleLanes - 1);
  const int64_t v = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / kScaleLanes;
  if (v >= n) return;   // a whole lane group
  float ws = 0.f;
  if (wsum) {
    ws = wsum[v];
  } else {
    const int32_t b = offsets[v], e = offsets[v + 1];
#pragma unroll 8
    for (int32_t j = b + lane; j < e; j += kScaleLanes) ws += entry_w[j];
#pragma unroll
    for (int o = kScaleLanes / 2; o > 0; o >>= 1) ws += __shfl_xor(ws, o, kScaleLanes);
  }
  const float scale = ws > 0.f ? 1.0f / ws : 0.f;
  for (int c = 4 * lane; c < C; c += 4 * kScaleLanes) {
    const float4 x = *reinterpret_cast<const float4*>(in + v * ld_in + c);
    *reinterpret_cast<float4*>(out + v * ld_out + c) = make_float4(x.x * scale, x.y * scale, x.z * scale, x.w * scale);
  }
}

// ---- convolution backward ----
// Taps 0 = self, 1..4 = +n_j, 5..8 = -n_j: the mirror of a tap negates its
// offset.
__device__ inline int mirror_tap(int t) { return t == 0 ? 0 : (t <= 4 ? t + 4 : t - 4); }

// Four values of a row of fp32 or bf16 elements (8-byte aligned for bf16).
template <bool BF16>
__device__ inline float4 load4(const void* base, int64_t at) {
  if constexpr (BF16) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + at);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(base) + at);
  }
}

// The two preparations of the convolution backward in one launch: the first
// mask_blocks workgroups write G = dY masked by Y > 0 (the forward's ReLU; 4
// channels per thread; bf16 values are masked as they are, so G stays
// exact), the rest write the adjoint convolution's weights Wt[t][i][o] =
// W[mirror t][o][i] (W laid out [tap][Cout][Cin]).  Either part may be empty.
template <bool BF16>
__global__ void __launch_bounds__(kBlock)
k_conv_bwd_prep(const void* __restrict__ dY, int64_t ld_dy, const void* __restrict__ Y, int64_t ld_y, int64_t n,
                void* __restrict__ G, int64_t ld_g, unsigned mask_blocks, const void* __restrict__ W, int Cout,
                int Cin, void* __restrict__ Wt) {
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  if (blockIdx.x < mask_blocks) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int c4 = Cout / 4;
    const int64_t v = q / c4;
    if (v >= n) return;
    const int c = 4 * static_cast<int>(q - v * c4);
    const E* d = static_cast<const E*>(dY) + v * ld_dy + c;
    const float4 y = load4<BF16>(Y, v * ld_y + c);
    E* g = static_cast<E*>(G) + v * ld_g + c;
    const bool on[4] = {y.x > 0.f, y.y > 0.f, y.z > 0.f, y.w > 0.f};
#pragma unroll
    for (int k = 0; k < 4; ++k) g[k] = on[k] ? d[k] : E(0);
    return;
  }
  const int64_t q = static_cast<int64_t>(blockIdx.x - mask_blocks) * kBlock + threadIdx.x;
  const int64_t per = static_cast<int64_t>(Cout) * Cin;
  if (q >= 9 * per) return;
  const int t = static_cast<int>(q / per);
  const int64_t r = q - t * per;
  const int i = static_cast<int>(r / Cout), o = static_cast<int>(r - static_cast<int64_t>(i) * Cout);
  static_cast<E*>(Wt)[q] = static_cast<const E*>(W)[(mirror_tap(t) * per) + static_cast<int64_t>(o) * Cin + i];
}

// dW[t][o][i] = sum_v G[v][o] X[nb(v,t)][i] as a GEMM with the vertices as
// the reduction dimension: A = G^T (Cout x K), B = the gathered rows
// (K x Cin); bf16 G and X are widened to fp32 as they are staged.  A workgroup owns one tap, one 64 x 64 tile of (o, i) and one
// chunk of V vertices; it stages 32 vertices at a time (G rows and gathered
// X rows, a missing neighbour reads as zeros) in double-buffered LDS, each
// wave multiplying a 32 x 32 sub-tile on v_mfma_f32_16x16x4_f32.  Partials
// go to part[chunk][tap][o][i]; the workgroups of tap 0 and the first i
// tile also sum the G columns (the bias gradient).
constexpr int kWgTile = 64;
constexpr int kWgStage = 32;
constexpr int kWgPitch = kWgTile + 4;

template <bool BF16>
__global__ void __launch_bounds__(kBlock)
k_conv_wgrad(const int32_t* __restrict__ nbr, int64_t ldn, int64_t n_out, int64_t V, const void* __restrict__ X,
             int64_t ld_x, int Cin, const void* __restrict__ G, int64_t ld_g, int Cout, int tiles_i,
             float* __restrict__ part, float* __restrict__ part_b) {
  __shared__ __align__(16) float Gs[2][kWgStage][kWgPitch];
  __shared__ __align__(16) float Xs[2][kWgStage][kWgPitch];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int64_t chunk = blockIdx.x;
  const int tap = blockIdx.y;
  const int ti = static_cast<int>(blockIdx.z) % tiles_i, to = static_cast<int>(blockIdx.z) / tiles_i;
  const int o0 = to * kWgTile, i0 = ti * kWgTile;
  const int64_t v_begin = chunk * V, v_end = min(v_begin + V, n_out);
  const int wo = (wave >> 1) * 32, wi = (wave & 1) * 32;
  const bool do_bias = part_b != nullptr && tap == 0 && ti == 0;
  const int lr = t >> 4, lc = 4 * (t & 15);   // rows lr and lr + 16, columns lc..lc+3 of a stage
  const int32_t* tab = nbr + static_cast<int64_t>(tap) * ldn;

  float4 ga[2], xa[2];
  auto load = [&](int64_t vb) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t v = vb + lr + 16 * h;
      float4 g = make_float4(0.f, 0.f, 0.f, 0.f), x = g;
      if (v < v_end) {
        if (o0 + lc < Cout) g = load4<BF16>(G, v * ld_g + o0 + lc);
        const int32_t u = tab[v];
        if (u >= 0 && i0 + lc < Cin) x = load4<BF16>(X, static_cast<int64_t>(u) * ld_x + i0 + lc);
      }
      ga[h] = g;
      xa[h] = x;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      *reinterpret_cast<float4*>(&Gs[buf][lr + 16 * h][lc]) = ga[h];
      *reinterpret_cast<float4*>(&Xs[buf][lr + 16 * h][lc]) = xa[h];
    }
  };

  f32x4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  float bsum = 0.f;

  load(v_begin);
  store(0);
  __syncthreads();
  int buf = 0;
  for (int64_t vb = v_begin; vb < v_end; vb += kWgStage) {
    const bool more = vb + kWgStage < v_end;
    if (more) load(vb + kWgStage);
#pragma unroll
    for (int ks = 0; ks < kWgStage / 4; ++ks) {
      float a[2], b[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        a[h] = Gs[buf][4 * ks + lg][wo + 16 * h + li];
        b[h] = Xs[buf][4 * ks + lg][wi + 16 * h + li];
      }
#pragma unroll
      for (int ao = 0; ao < 2; ++ao)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) acc[ao][bi] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[ao], b[bi], acc[ao][bi], 0, 0, 0);
    }
    if (do_bias && t < kWgTile)
#pragma unroll 8
      for (int r = 0; r < kWgStage; ++r) bsum += Gs[buf][r][t];
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // lane (i, g) of block (ao, bi) holds o = 16 ao + 4 g + r, i = 16 bi + i
  float* P = part + (chunk * 9 + tap) * static_cast<int64_t>(Cout) * Cin;
#pragma unroll
  for (int ao = 0; ao < 2; ++ao)
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = o0 + wo + 16 * ao + 4 * lg + r, i = i0 + wi + 16 * bi + li;
        if (o < Cout && i < Cin) P[static_cast<int64_t>(o) * Cin + i] = acc[ao][bi][r];
      }
  if (do_bias && t < kWgTile && o0 + t < Cout) part_b[chunk * Cout + o0 + t] = bsum;
}

// dW = sum over chunks of the partials, dbias likewise; fixed order.  A
// thread sums 4 consecutive entries (count and Cout are multiples of 4).
__global__ void __launch_bounds__(kBlock)
k_wgrad_reduce(const float* __restrict__ part, const float* __restrict__ part_b, int64_t chunks, int64_t count,
               int Cout, float* __restrict__ dW, float* __restrict__ dbias) {
  const int64_t q = 4 * (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x);
  const float* src;
  int64_t stride;
  float* dst;
  if (q < count) {
    src = part + q;
    stride = count;
    dst = dW ? dW + q : nullptr;
  } else if (q < count + Cout) {
    src = part_b + (q - count);
    stride = Cout;
    dst = dbias ? dbias + (q - count) : nullptr;
  } else {
    return;
  }
  if (!dst) return;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int64_t c = 0; c < chunks; ++c) {
    const float4 x = *reinterpret_cast<const float4*>(src + c * stride);
    a.x += x.x;
    a.y += x.y;
    a.z += x.z;
    a.w += x.w;
  }
  *reinterpret_cast<float4*>(dst) = a;
}

inline unsigned blocks_for(int64_t threads) { return static_cast<unsigned>((threads + kBlock - 1) / kBlock); }

// Vertex chunks of the weight gradient: about two workgroups per compute
// unit over taps and tiles (more chunks would only grow the partials the
// reduction reads), chunks a multiple of the stage.
void wgrad_chunks(int64_t n_out, int tiles, int64_t* chunks, int64_t* V) {
  int64_t want = std::max<int64_t>(1, 512 / (9 * static_cast<int64_t>(tiles)));
  want = std::min<int64_t>(want, (n_out + kWgStage - 1) / kWgStage);
  int64_t v = (n_out + want - 1) / want;
  v = (v + kWgStage - 1) / kWgStage * kWgStage;
  *V = v;
  *chunks = (n_out + v - 1) / v;
}


// ---- linear layers backward (the classifier fused with DeformSlice, the
// 1x1 layers of Distribute + PointNet) ----
// For out_p = W a_p + b over rows p (W: K x C, [out][in]) and G = dL/dout:
//   dA_p = sum_j G_pj W[j]   (k_lin_dinput),
//   dW = sum_p G_p a_p^T, db = sum_p G_p   (k_lin_wgrad over chunks of rows,
//   then k_lin_reduce adds the chunks' partials in chunk order).
// a_p is either given or max(x_p scale + shift, 0) of given rows x_p (the
// pre-activation table pre = [C scales][C shifts]).
constexpr int kClsPts = 32;        // rows staged per step of k_lin_wgrad
constexpr int kClsMaxChunks = 1024;

// dA_p[c] = sum_j G_pj W[j][c]: one thread per (row, 4 channels).
__global__ void __launch_bounds__(kBlock)
k_lin_dinput(const float* __restrict__ z, int64_t ld_z, const float* __restrict__ Wc, int K, int C, int64_t m,
             float* __restrict__ df, int64_t ld_df) {
  const int quads = C / 4;
  const int64_t total = m * quads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t p = i / quads;
    const int c = 4 * static_cast<int>(i - p * quads);
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < K; ++j) {
      const float zj = z[p * ld_z + j];
      const float4 w = *reinterpret_cast<const float4*>(Wc + static_cast<int64_t>(j) * C + c);
      a.x = fmaf(zj, w.x, a.x);
      a.y = fmaf(zj, w.y, a.y);
      a.z = fmaf(zj, w.z, a.z);
      a.w = fmaf(zj, w.w, a.w);
    }
    *reinterpret_cast<float4*>(df + p * ld_df + c) = a;
  }
}

// Workgroup w: over its chunk of rows, part[w][j C + c] = sum_p G_pj a_pc and
// part[w][K C + j] = sum_p G_pj, rows in order; rows of G and a are staged
// kClsPts at a time in LDS (a pre-activated as they are staged when pre is
// given).  Thread t owns outputs t, t + 256, ...
template <int NO>
__global__ void __launch_bounds__(kBlock)
k_lin_wgrad(const float* __restrict__ z, int64_t ld_z, const float* __restrict__ f, int64_t ld_f,
            const float* __restrict__ pre, int K, int C, int64_t m, int64_t chunk, float* __restrict__ part) {
  extern __shared__ float sm[];
  float* sz = sm;                    // [kClsPts][K]
  float* sf = sm + kClsPts * K;      // [kClsPts][C]
  const int t = threadIdx.x;
  const int nout = K * C + K;
  const int64_t p0 = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t p1 = min(p0 + chunk, m);
  float acc[NO];
#pragma unroll
  for (int k = 0; k < NO; ++k) acc[k] = 0.f;
  for (int64_t pb = p0; pb < p1; pb += kClsPts) {
    const int np = static_cast<int>(min<int64_t>(kClsPts, p1 - pb));
    __syncthreads();
    for (int e = t; e < np * K; e += kBlock) sz[e] = z[(pb + e / K) * ld_z + e % K];
    for (int e = t; e < np * (C / 4); e += kBlock) {
      const int r = e / (C / 4), q = e - r * (C / 4);
      float4 v = *reinterpret_cast<const float4*>(f + (pb + r) * ld_f + 4 * q);
      if (pre) {
        v.x = fmaxf(fmaf(v.x, pre[4 * q], pre[C + 4 * q]), 0.f);
        v.y = fmaxf(fmaf(v.y, pre[4 * q + 1], pre[C + 4 * q + 1]), 0.f);
        v.z = fmaxf(fmaf(v.z, pre[4 * q + 2], pre[C + 4 * q + 2]), 0.f);
        v.w = fmaxf(fmaf(v.w, pre[4 * q + 3], pre[C + 4 * q + 3]), 0.f);
      }
      *reinterpret_cast<float4*>(sf + r * C + 4 * q) = v;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NO; ++k) {
      const int o = t + k * kBlock;
      if (o >= nout) break;
      float a = acc[k];
      if (o < K * C) {
        const int j = o / C, c = o - j * C;
        for (int r = 0; r < np; ++r) a = fmaf(sz[r * K + j], sf[r * C + c], a);
      } else {
        for (int r = 0; r < np; ++r) a += sz[r * K + (o - K * C)];
      }
      acc[k] = a;
    }
  }
  float* dst = part + static_cast<int64_t>(blockIdx.x) * nout;
#pragma unroll
  for (int k = 0; k < NO; ++k)
    if (t + k * kBlock < nout) dst[t + k * kBlock] = acc[k];
}

// dW[j][c] (c < C_out, row stride C_out) and db[j]: sums over the chunks of
// part[w][o], in chunk order.
__global__ void __launch_bounds__(kBlock)
k_lin_reduce(const float* __restrict__ part, int chunks, int K, int C, int C_out, float* __restrict__ dWc,
             float* __restrict__ dbc) {
  const int nout = K * C + K;
  const int o = blockIdx.x * kBlock + threadIdx.x;
  if (o >= nout) return;
  float a = 0.f;
  for (int w = 0; w < chunks; ++w) a += part[static_cast<int64_t>(w) * nout + o];
  if (o < K * C) {
    const int j = o / C, c = o - j * C;
    if (dWc && c < C_out) dWc[j * C_out + c] = a;
  } else if (dbc) {
    dbc[o - K * C] = a;
  }
}

void cls_chunks(int64_t m, int64_t* chunk, int* chunks) {
  int64_t c = std::max<int64_t>(kClsPts, (m + kClsMaxChunks - 1) / kClsMaxChunks);
  c = (c + kClsPts - 1) / kClsPts * kClsPts;
  *chunk = c;
  *chunks = static_cast<int>(std::max<int64_t>(1, (m + c - 1) / c));
}

}  // namespace

void launch_scale_by_weight_sum(const int32_t* offsets, const float* entry_w, const float* wsum, int64_t n,
                                const float* in, int64_t ld_in, int C, float* out, int64_t ld_out, hipStream_t s) {
  if (n <= 0) return;
  launch(k_scale_by_weight_sum, dim3(blocks_for(n * kScaleLanes)), dim3(kBlock), 0, s, offsets, entry_w, wsum, n, in,
         ld_in, C, out, ld_out);
}

void launch_conv_bwd_prep(const void* dY, int64_t ld_dy, const void* Y, int64_t ld_y, int64_t n, void* G,
                          int64_t ld_g, const void* W, int Cout, int Cin, void* Wt, int bf16, hipStream_t s) {
  const unsigned mb = (G && n > 0) ? blocks_for(n * (Cout / 4)) : 0;
  const unsigned wb = Wt ? blocks_for(9LL * Cout * Cin) : 0;
  if (mb + wb == 0) return;
  if (bf16)
    launch(k_conv_bwd_prep<true>, dim3(mb + wb), dim3(kBlock), 0, s, dY, ld_dy, Y, ld_y, n, G, ld_g, mb, W, Cout, Cin,
           Wt);
  else
    launch(k_conv_bwd_prep<false>, dim3(mb + wb), dim3(kBlock), 0, s, dY, ld_dy, Y, ld_y, n, G, ld_g, mb, W, Cout, Cin,
           Wt);
}

int64_t wgrad_partial_floats(int64_t n_out, int Cout, int Cin) {
  if (n_out <= 0) return 0;
  const int tiles = ((Cout + kWgTile - 1) / kWgTile) * ((Cin + kWgTile - 1) / kWgTile);
  int64_t chunks, V;
  wgrad_chunks(n_out, tiles, &chunks, &V);
  return chunks * (9LL * Cout * Cin + Cout);
}

void launch_conv_wgrad(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* X, int64_t ld_x, int Cin,
                       const void* G, int64_t ld_g, int Cout, float* dW, float* dbias, float* partials, int bf16,
                       hipStream_t s) {
  const int tiles_o = (Cout + kWgTile - 1) / kWgTile, tiles_i = (Cin + kWgTile - 1) / kWgTile;
  const int64_t count = 9LL * Cout * Cin;
  int64_t chunks = 0, V = 0;
  if (n_out > 0) wgrad_chunks(n_out, tiles_o * tiles_i, &chunks, &V);
  float* part = partials;
  float* part_b = dbias ? partials + chunks * count : nullptr;
  if (chunks > 0) {
    const dim3 grid(static_cast<unsigned>(chunks), 9, static_cast<unsigned>(tiles_o * tiles_i));
    if (bf16)
      launch(k_conv_wgrad<true>, grid, dim3(kBlock), 0, s, nbr, ldn, n_out, V, X, ld_x, Cin, G, ld_g, Cout, tiles_i,
             part, part_b);
    else
      launch(k_conv_wgrad<false>, grid, dim3(kBlock), 0, s, nbr, ldn, n_out, V, X, ld_x, Cin, G, ld_g, Cout, tiles_i,
             part, part_b);
  }
  // with no output vertex (chunks = 0) the sums below are zero
  launch(k_wgrad_reduce, dim3(blocks_for((count + Cout) / 4)), dim3(kBlock), 0, s, static_cast<const float*>(part),
         static_cast<const float*>(part_b), chunks, count, Cout, dW, dbias);
}

}  // namespace lat

namespace lat {

int64_t classify_backward_partial_floats(int64_t m, int K, int C) {
  int64_t chunk;
  int chunks;
  cls_chunks(m, &chunk, &chunks);
  return static_cast<int64_t>(chunks) * (static_cast<int64_t>(K) * C + K);
}

void launch_linear_backward(const float* z, int64_t ld_z, const float* W, int K, int C, int64_t m, const float* f,
                            int64_t ld_f, const float* pre, float* df, int64_t ld_df, float* dW, int C_out, float* db,
                            float* part, hipStream_t s) {
  if (df && m > 0) {
    const int64_t b = (m * (C / 4) + kBlock - 1) / kBlock;
    launch(k_lin_dinput, dim3(static_cast<unsigned>(std::min<int64_t>(b, 8192))), dim3(kBlock), 0, s, z, ld_z, W, K,
           C, m, df, ld_df);
  }
  if (!dW && !db) return;
  const int nout = K * C + K;
  int64_t chunk;
  int chunks;
  cls_chunks(m, &chunk, &chunks);
  if (m > 0) {
    const size_t lds = sizeof(float) * kClsPts * static_cast<size_t>(K + C);
    auto go = [&](auto no_c) {
      constexpr int NO = decltype(no_c)::value;
      static bool lds_limit_set = false;
      if (!lds_limit_set) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_lin_wgrad<NO>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(sizeof(float) * kClsPts * (64 + 512)));
        lds_limit_set = true;
      }
      launch(k_lin_wgrad<NO>, dim3(static_cast<unsigned>(chunks)), dim3(kBlock), static_cast<uint32_t>(lds), s, z,
             ld_z, f, ld_f, pre, K, C, m, chunk, part);
    };
    const int no = (nout + kBlock - 1) / kBlock;
    if (no <= 2) go(std::integral_constant<int, 2>{});
    else if (no <= 8) go(std::integral_constant<int, 8>{});
    else if (no <= 24) go(std::integral_constant<int, 24>{});
    else go(std::integral_constant<int, 65>{});
  }
  launch(k_lin_reduce, dim3(static_cast<unsigned>((nout + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
         static_cast<const float*>(part), m > 0 ? chunks : 0, K, C, C_out, dW, db);
}

void launch_classify_backward(const float* z, int64_t ld_z, const float* Wc, int K, int C, int64_t m, const float* f,
                              float* df, float* dWc, float* dbc, float* part, hipStream_t s) {
  ScopedKernelTimer tm("classify_bwd", s);
  launch_linear_backward(z, ld_z, Wc, K, C, m, f, C, nullptr, df, C, dWc, C, dbc, part, s);
}

}  // namespace lat

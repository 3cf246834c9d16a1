// Distribute + PointNet on gfx950 (Proposed Operations, Eq. (distribute),
// and the PointNet block of the architecture figure):
//   x_v = max_{p in J_v} W3 relu(W2 relu(W1 [g_p - mu_v ; f_p] + b1) + b2) + b3,
//   mu_v = mean of g_p over J_v.
// J_v are the vertex lists built with the lattice (entries grouped by vertex).
// Both per-vertex reductions (the mean and the maximum) run over spans of
// consecutive list entries, so the work is balanced however skewed the list
// lengths are: a vertex inside a span is finished there; the vertex a span
// starts inside and the vertex that runs past its end leave a head and a tail
// partial, which a finishing pass joins in span order.  The mean is summed in
// fp64 (positions can be tens of metres from the origin while g - mu is a
// fraction of sigma) and g - mu is rounded to fp32 once; the three 1x1
// layers run on v_mfma_f32_16x16x4_f32, 16 list entries per wave.
#include <algorithm>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int kMeanSpan = kBlock;  // list entries per workgroup of the mean pass
constexpr int kMlpSpan = 64;       // list entries per workgroup of the MLP pass (16 per wave)
constexpr int kMaxC = 64;          // widest 1x1 layer

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Offsets of the vertices whose lists overlap [s0, s0 + span): the window
// starts at the vertex owning position s0 (chunk_first, span a multiple of
// the chunk) and holds span + 2 list ends, clamped to n.
__device__ inline void load_window(const int32_t* __restrict__ offsets, int64_t n, int32_t v0, int count,
                                   int32_t* win) {
  for (int i = threadIdx.x; i < count; i += blockDim.x) {
    const int64_t v = min(static_cast<int64_t>(v0) + i, n);
    win[i] = offsets[v];
  }
}

// Index in the window of the vertex whose list holds position s:
// the largest j with win[j] <= s.
__device__ inline int window_vertex(const int32_t* win, int count, int64_t s) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (win[mid] <= s) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// ---- mean of the positions over J_v (fp64) ----
__global__ void __launch_bounds__(kBlock)
k_dist_mean(const int32_t* __restrict__ offsets, const int32_t* __restrict__ entries,
            const int32_t* __restrict__ chunk_first, int chunk, int64_t n, int64_t total,
            const float* __restrict__ pos, double4* __restrict__ mu, double4* __restrict__ part_head,
            double4* __restrict__ part_tail) {
  constexpr int W = kMeanSpan + 2;
  __shared__ int32_t win[W];
  __shared__ double sx[2][kBlock], sy[2][kBlock], sz[2][kBlock];
  __shared__ int32_t sf[2][kBlock];
  const int t = threadIdx.x;
  const int64_t span = blockIdx.x;
  const int64_t s0 = span * kMeanSpan;
  const int64_t s1 = min(s0 + kMeanSpan, total);
  const int32_t v0 = chunk_first[s0 / chunk];
  load_window(offsets, n, v0, W, win);
  __syncthreads();
  const int64_t s = s0 + t;
  const bool live = s < s1;
  int vi = 0;
  double x = 0.0, y = 0.0, z = 0.0;
  if (live) {
    vi = window_vertex(win, W, s);
    const int64_t p = entries[s] >> 2;
    x = pos[3 * p];
    y = pos[3 * p + 1];
    z = pos[3 * p + 2];
  }
  // segmented inclusive scan (Hillis-Steele, fixed order): a segment starts
  // where a vertex's list starts or at the span's first entry
  int flag = (t == 0 || (live && win[vi] == s)) ? 1 : 0;
  int cur = 0;
  sx[cur][t] = x; sy[cur][t] = y; sz[cur][t] = z; sf[cur][t] = flag;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    const int nxt = cur ^ 1;
    double ax = sx[cur][t], ay = sy[cur][t], az = sz[cur][t];
    int af = sf[cur][t];
    if (t >= off && !af) {
      ax += sx[cur][t - off];
      ay += sy[cur][t - off];
      az += sz[cur][t - off];
      af = sf[cur][t - off];
    } else if (t >= off) {
      af = 1;
    }
    sx[nxt][t] = ax; sy[nxt][t] = ay; sz[nxt][t] = az; sf[nxt][t] = af;
    __syncthreads();
    cur = nxt;
  }
  if (!live) return;
  const int64_t vb = win[vi], ve = win[vi + 1];
  if (s + 1 != min(ve, s1)) return;            // not the last entry of its piece
  const double4 sum = make_double4(sx[cur][t], sy[cur][t], sz[cur][t], 0.0);
  if (vb >= s0 && ve <= s1) {
    const double inv = 1.0 / static_cast<double>(ve - vb);
    mu[v0 + vi] = make_double4(sum.x * inv, sum.y * inv, sum.z * inv, 0.0);
  } else if (vb < s0) {
    part_head[span] = sum;
  } else {
    part_tail[span] = sum;
  }
}

// Vertices cut by span boundaries: the span where a vertex starts adds its
// tail partial and the head partials of the following spans, in order.
__global__ void __launch_bounds__(kBlock)
k_dist_mean_finish(const int32_t* __restrict__ offsets, const int32_t* __restrict__ chunk_first, int chunk,
                   int64_t nspans, double4* __restrict__ mu, const double4* __restrict__ part_head,
                   const double4* __restrict__ part_tail) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (c + 1 >= nspans) return;
  const int64_t s0 = c * kMeanSpan, s1 = s0 + kMeanSpan;
  const int32_t v = chunk_first[s1 / chunk];
  const int64_t vb = offsets[v];
  if (!(vb >= s0 && vb < s1)) return;
  const int64_t ve = offsets[v + 1];
  const int64_t last = (ve - 1) / kMeanSpan;
  double4 a = part_tail[c];
  for (int64_t c2 = c + 1; c2 <= last; ++c2) {
    const double4 h = part_head[c2];
    a.x += h.x; a.y += h.y; a.z += h.z;
  }
  const double inv = 1.0 / static_cast<double>(ve - vb);
  mu[v] = make_double4(a.x * inv, a.y * inv, a.z * inv, 0.0);
}

// ---- the three 1x1 layers and the maximum over J_v ----
// LDS: weights as [k][n] (n contiguous) for the B operand, per-wave input
// rows X (16 x K1), per-wave hidden rows H (16 x max(C1, C2)) twice, and the
// workgroup's output rows (64 x C3).
struct MlpLds {
  int k1, c1, c2, c3;
  int ldx, ldh, ldo, ld1, ld2, ld3;
  size_t w1, w2, w3, b, x, h1, h2, o, win, rows, end;
  __host__ __device__ MlpLds(int K1, int C1, int C2, int C3) : k1(K1), c1(C1), c2(C2), c3(C3) {
    // every row pitch is odd, so the 4 k rows read by one MFMA operand load
    // fall in different LDS banks
    ldx = K1 + 1;
    ldh = (C1 > C2 ? C1 : C2) + 1;
    ldo = C3 + 1;
    ld1 = C1 + 1;
    ld2 = C2 + 1;
    ld3 = C3 + 1;
    w1 = 0;
    w2 = w1 + static_cast<size_t>(K1) * ld1;
    w3 = w2 + static_cast<size_t>(C1) * ld2;
    b = w3 + static_cast<size_t>(C2) * ld3;
    x = b + C1 + C2 + C3;
    h1 = x + 4 * 16 * static_cast<size_t>(ldx);
    h2 = h1 + 4 * 16 * static_cast<size_t>(ldh);
    o = h2 + 4 * 16 * static_cast<size_t>(ldh);
    win = o + kMlpSpan * static_cast<size_t>(ldo);   // int32 from here on
    rows = win + kMlpSpan + 2;                         // per entry: point, window index, end code
    end = rows + 3 * kMlpSpan;
  }
  __host__ __device__ size_t bytes() const { return end * 4; }
};

// One 16 x 16 output tile of a wave: sum over k of A[16 x K] (LDS, row
// pitch lda) times B[K x N] (LDS, [k][n], pitch ldb) for columns n0..n0+15.
__device__ inline f32x4 tile_mma(const float* A, int lda, const float* B, int ldb, int K, int n0, int lane) {
  const int li = lane & 15, lg = lane >> 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < K; k0 += 4)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A[li * lda + k0 + lg], B[(k0 + lg) * ldb + n0 + li], acc, 0, 0, 0);
  return acc;
}

// Persistent: a workgroup stages the weights once and takes spans
// blockIdx.x, blockIdx.x + gridDim.x, ...
__global__ void __launch_bounds__(kBlock)
k_dist_mlp(const int32_t* __restrict__ offsets, const int32_t* __restrict__ entries,
           const int32_t* __restrict__ chunk_first, int chunk, int64_t n, int64_t total,
           const float* __restrict__ pos, const float* __restrict__ feat, int64_t ld_feat, int cf,
           const double4* __restrict__ mu, const float* __restrict__ W1, const float* __restrict__ b1,
           const float* __restrict__ W2, const float* __restrict__ b2, const float* __restrict__ W3,
           const float* __restrict__ b3, int K1, int C1, int C2, int C3, float* __restrict__ out,
           int64_t ld_out, float* __restrict__ part_head, float* __restrict__ part_tail, int64_t nspans) {
  extern __shared__ __align__(16) float sm[];
  const MlpLds lay(K1, C1, C2, C3);
  float* w1 = sm + lay.w1;
  float* w2 = sm + lay.w2;
  float* w3 = sm + lay.w3;
  float* bs = sm + lay.b;
  int32_t* win = reinterpret_cast<int32_t*>(sm + lay.win);
  int32_t* rp = reinterpret_cast<int32_t*>(sm + lay.rows);   // point of each entry
  int32_t* rv = rp + kMlpSpan;                                // window index of its vertex
  int32_t* rc = rv + kMlpSpan;                                // end code: -1, or 4 * window index + kind
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int li = lane & 15, lg = lane >> 4;
  constexpr int W = kMlpSpan + 2;

  // weights, transposed to [k][n]; input k of the first layer: 0..2 the
  // coordinates, 3 a zero pad, 4.. the features
  const int cin = 3 + cf;
  for (int i = t; i < K1 * C1; i += kBlock) {
    const int k = i / C1, o = i - k * C1;
    const int src = k < 3 ? k : (k == 3 ? -1 : (k - 4 < cf ? k - 1 : -1));
    w1[k * lay.ld1 + o] = src >= 0 ? W1[o * cin + src] : 0.f;
  }
  for (int i = t; i < C1 * C2; i += kBlock) {
    const int k = i / C2, o = i - k * C2;
    w2[k * lay.ld2 + o] = W2[o * C1 + k];
  }
  for (int i = t; i < C2 * C3; i += kBlock) {
    const int k = i / C3, o = i - k * C3;
    w3[k * lay.ld3 + o] = W3[o * C2 + k];
  }
  for (int i = t; i < C1 + C2 + C3; i += kBlock) {
    float v = 0.f;
    if (i < C1) v = b1 ? b1[i] : 0.f;
    else if (i < C1 + C2) v = b2 ? b2[i - C1] : 0.f;
    else v = b3 ? b3[i - C1 - C2] : 0.f;
    bs[i] = v;
  }
  float* X = sm + lay.x + wave * 16 * lay.ldx;
  float* H1 = sm + lay.h1 + wave * 16 * lay.ldh;
  float* H2 = sm + lay.h2 + wave * 16 * lay.ldh;
  float* O = sm + lay.o;

  for (int64_t span = blockIdx.x; span < nspans; span += gridDim.x) {
    const int64_t s0 = span * kMlpSpan;
    const int64_t s1 = min(s0 + kMlpSpan, total);
    const int32_t v0 = chunk_first[s0 / chunk];
    __syncthreads();   // the previous span is done with the LDS rows
    load_window(offsets, n, v0, W, win);
    __syncthreads();
    if (t < kMlpSpan) {
      const int64_t s = s0 + t;
      int32_t p = -1, vi = 0, code = -1;
      if (s < s1) {
        p = entries[s] >> 2;
        vi = window_vertex(win, W, s);
        const int64_t vb = win[vi], ve = win[vi + 1];
        if (s + 1 == min(ve, s1)) code = 4 * vi + ((vb >= s0 && ve <= s1) ? 0 : (vb < s0 ? 1 : 2));
      }
      rp[t] = p;
      rv[t] = vi;
      rc[t] = code;
    }
    __syncthreads();

    // input rows of this wave's 16 entries: [g - mu (fp64, rounded once), 0, f]
    for (int i = lane; i < 16 * K1; i += 64) {
      const int r = i / K1, k = i - r * K1;
      const int e = wave * 16 + r;
      const int32_t p = rp[e];
      float v = 0.f;
      if (p >= 0) {
        if (k < 3) {
          const double4 m = mu[v0 + rv[e]];
          const double mk = k == 0 ? m.x : (k == 1 ? m.y : m.z);
          v = static_cast<float>(static_cast<double>(pos[3 * static_cast<int64_t>(p) + k]) - mk);
        } else if (k >= 4 && k - 4 < cf) {
          v = feat[static_cast<int64_t>(p) * ld_feat + (k - 4)];
        }
      }
      X[r * lay.ldx + k] = v;
    }
    // X, H1 and H2 are this wave's own rows: LDS accesses of one wave take
    // effect in order, so a wave-level fence (no workgroup barrier) orders
    // each layer's writes before the next layer's reads
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // layer 1, ReLU applied when the rows are read by layer 2
    for (int n0 = 0; n0 < C1; n0 += 16) {
      const f32x4 a = tile_mma(X, lay.ldx, w1, lay.ld1, K1, n0, lane);
      for (int r = 0; r < 4; ++r) H1[(4 * lg + r) * lay.ldh + n0 + li] = fmaxf(a[r] + bs[n0 + li], 0.f);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int n0 = 0; n0 < C2; n0 += 16) {
      const f32x4 a = tile_mma(H1, lay.ldh, w2, lay.ld2, C1, n0, lane);
      for (int r = 0; r < 4; ++r) H2[(4 * lg + r) * lay.ldh + n0 + li] = fmaxf(a[r] + bs[C1 + n0 + li], 0.f);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int n0 = 0; n0 < C3; n0 += 16) {
      const f32x4 a = tile_mma(H2, lay.ldh, w3, lay.ld3, C2, n0, lane);
      for (int r = 0; r < 4; ++r)
        O[(wave * 16 + 4 * lg + r) * lay.ldo + n0 + li] = a[r] + bs[C1 + C2 + n0 + li];
    }
    __syncthreads();

    // per-channel maximum over each vertex's rows in the span; the end codes
    // mark the last row of every vertex's piece
    if (t < C3) {
      const int rows = static_cast<int>(s1 - s0);
      float m = -INFINITY;
#pragma unroll 8
      for (int e = 0; e < rows; ++e) {
        m = fmaxf(m, O[e * lay.ldo + t]);
        const int32_t code = rc[e];
        if (code < 0) continue;
        const int kind = code & 3, vi = code >> 2;
        if (kind == 0) out[static_cast<int64_t>(v0 + vi) * ld_out + t] = m;
        else if (kind == 1) part_head[span * C3 + t] = m;
        else part_tail[span * C3 + t] = m;
        m = -INFINITY;
      }
    }
  }
}

__global__ void __launch_bounds__(kBlock)
k_dist_max_finish(const int32_t* __restrict__ offsets, const int32_t* __restrict__ chunk_first, int chunk,
                  int64_t nspans, int C3, float* __restrict__ out, int64_t ld_out,
                  const float* __restrict__ part_head, const float* __restrict__ part_tail) {
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int64_t c = g / C3;
  const int ch = static_cast<int>(g - c * C3);
  if (c + 1 >= nspans) return;
  const int64_t s0 = c * kMlpSpan, s1 = s0 + kMlpSpan;
  const int32_t v = chunk_first[s1 / chunk];
  const int64_t vb = offsets[v];
  if (!(vb >= s0 && vb < s1)) return;
  const int64_t ve = offsets[v + 1];
  const int64_t last = (ve - 1) / kMlpSpan;
  float m = part_tail[c * C3 + ch];
  for (int64_t c2 = c + 1; c2 <= last; ++c2) m = fmaxf(m, part_head[c2 * C3 + ch]);
  out[static_cast<int64_t>(v) * ld_out + ch] = m;
}

}  // namespace

int64_t distribute_workspace_bytes(int64_t total, int C3) {
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  const int64_t mlp_spans = (total + kMlpSpan - 1) / kMlpSpan;
  return 2 * mean_spans * static_cast<int64_t>(sizeof(double4)) + 2 * mlp_spans * C3 * 4;
}

int distribute_max_features() { return kMaxC - 4; }

void launch_distribute(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                       int64_t n, int64_t total, const float* pos, const float* feat, int64_t ld_feat, int cf,
                       const float* W1, const float* b1, int C1, const float* W2, const float* b2, int C2,
                       const float* W3, const float* b3, int C3, float* out, int64_t ld_out, double* mu,
                       void* work, hipStream_t s) {
  if (total <= 0 || n <= 0) return;
  ScopedKernelTimer tm("distribute", s);
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  const int64_t mlp_spans = (total + kMlpSpan - 1) / kMlpSpan;
  double4* mh = static_cast<double4*>(work);
  double4* mt = mh + mean_spans;
  float* ph = reinterpret_cast<float*>(mt + mean_spans);
  float* pt = ph + mlp_spans * C3;
  double4* mu4 = reinterpret_cast<double4*>(mu);
  launch(k_dist_mean, dim3(static_cast<unsigned>(mean_spans)), dim3(kBlock), 0, s, offsets, entries, chunk_first,
         chunk, n, total, pos, mu4, mh, mt);
  if (mean_spans > 1)
    launch(k_dist_mean_finish, dim3(static_cast<unsigned>((mean_spans + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
           offsets, chunk_first, chunk, mean_spans, mu4, static_cast<const double4*>(mh),
           static_cast<const double4*>(mt));
  const int K1 = ((3 + cf) + 1 + 3) / 4 * 4;   // coordinates, a zero pad, features; multiple of 4
  const MlpLds lay(K1, C1, C2, C3);
  static bool lds_limit_set = false;
  if (!lds_limit_set) {
    const MlpLds worst(kMaxC, kMaxC, kMaxC, kMaxC);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_dist_mlp), hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(worst.bytes()));
    lds_limit_set = true;
  }
  const unsigned grid = static_cast<unsigned>(std::min<int64_t>(mlp_spans, 2048));
  launch(k_dist_mlp, dim3(grid), dim3(kBlock), static_cast<uint32_t>(lay.bytes()), s, offsets, entries, chunk_first,
         chunk, n, total, pos, feat, ld_feat, cf, static_cast<const double4*>(mu4), W1, b1, W2, b2, W3, b3, K1, C1, C2,
         C3, out, ld_out, ph, pt, mlp_spans);
  if (mlp_spans > 1) {
    const int64_t threads = mlp_spans * C3;
    launch(k_dist_max_finish, dim3(static_cast<unsigned>((threads + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
           offsets, chunk_first, chunk, mlp_spans, C3, out, ld_out, static_cast<const float*>(ph),
           static_cast<const float*>(pt));
  }
}

}  // namespace lat

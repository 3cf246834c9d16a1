// Distribute + PointNet on gfx950 (Proposed Operations, Eq. (distribute),
// the scaled positions G_s = G / sigma of the Method section, and the
// PointNet block of the architecture figure):
//   r = [g_p / sigma - mu_v ; f_p] for every p in J_v, mu_v = mean of g_p / sigma over J_v,
//   h_i = W_i relu(GN_i(h_{i-1})) + b_i  (h_0 = r, i = 1..3),  x_v = max over J_v of h_3.
// GroupNorm's statistics span all distributed rows; a layer of at most 32
// channels has one channel per group, a wider one 32 groups.
// J_v are the vertex lists built with the lattice (entries grouped by vertex).
// The mean runs over spans of 256 consecutive list entries, so the work is
// balanced however skewed the list lengths are: a vertex inside a span is
// finished there; the vertex a span starts inside and the vertex that runs
// past its end leave a head and a tail partial, which a finishing pass joins
// in span order.  The mean is summed in fp64 (positions can be hundreds of
// sigma from the origin while g - mu is a fraction of one) and g - mu is
// rounded to fp32 once.  Each normalisation needs the statistics of its
// whole input before any row can pass it, so the rows are walked four
// times: the statistics of r, then of h_1 and of h_2 (each pass recomputes
// the cheaper layers before it rather than storing them), then the full
// block with the maximum.  Statistics are fp64 per-workgroup partials added
// in a fixed order, so the result does not depend on scheduling.  The 1x1
// layers run on v_mfma_f32_16x16x4_f32 with the activations held in
// registers; each wave takes an equal range of list entries and reduces
// the maximum across lanes.
#include <algorithm>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int kMeanSpan = kBlock;  // list entries per workgroup of the mean pass
constexpr int kMaxC = 64;          // widest 1x1 layer
constexpr int kMaxIn = 32;         // widest raw row (d + Cf): one channel per normalisation group
constexpr int kPreStride = 2 * kMaxC;   // floats per normalisation table: scales, then shifts
constexpr int kStatsMaxParts = 2048;    // partials of the raw-row statistics

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

// ---- mean of the positions over J_v (fp64, in units of sigma) ----
__global__ void __launch_bounds__(kBlock)
k_dist_mean(const int32_t* __restrict__ offsets, const int32_t* __restrict__ entries,
            const int32_t* __restrict__ chunk_first, int chunk, int64_t n, int64_t total,
            const float* __restrict__ pos, double sc0, double sc1, double sc2, double4* __restrict__ mu,
            double4* __restrict__ part_head, double4* __restrict__ part_tail, int32_t* __restrict__ entry_vertex,
            int64_t R, float* __restrict__ out, int64_t ld_out, int C3) {
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
    entry_vertex[s] = v0 + vi;
    const int64_t p = entries[s] >> 2;
    x = static_cast<double>(pos[3 * p]) / sc0;
    y = static_cast<double>(pos[3 * p + 1]) / sc1;
    z = static_cast<double>(pos[3 * p + 2]) / sc2;
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
  if (vb >= s0 && (ve - 1) / R != vb / R) {
    // the list is cut by a range boundary of the MLP pass, whose maximum
    // over it is then taken atomically into this row
    float* o = out + static_cast<int64_t>(v0 + vi) * ld_out;
    for (int c = 0; c < C3; ++c) o[c] = -INFINITY;
  }
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

// Coordinate c (< 3) of the distributed row of entry (point p, vertex mean m):
// g / sigma - mu in fp64, rounded to fp32 once.  The statistics pass and the
// MLP passes form it by this one expression, so they see the same rows.
__device__ inline float row_coord(float g, double sc, double m) {
  return static_cast<float>(static_cast<double>(g) / sc - m);
}

// ---- statistics of the raw distributed rows (first normalisation) ----
// Thread t of workgroup w takes the entries w * 256 + t, + 256 * grid, ...,
// and sums channels [c0, c0 + 8) of their rows (for each block of 8 of the
// cin channels in turn); the workgroup adds its 256 threads by a fixed tree.
// part[w] holds the cin sums, then the cin sums of squares.
constexpr int kStatsCh = 8;
__global__ void __launch_bounds__(kBlock)
k_dist_in_stats(const int32_t* __restrict__ entries, const int32_t* __restrict__ entry_vertex, int64_t total,
                const float* __restrict__ pos, double sc0, double sc1, double sc2, const double4* __restrict__ mu,
                const float* __restrict__ feat, int64_t ld_feat, int cin, double* __restrict__ part) {
  __shared__ double sh[2][kBlock];
  const int t = threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int c0 = 0; c0 < cin; c0 += kStatsCh) {
    double s[kStatsCh], ss[kStatsCh];
#pragma unroll
    for (int i = 0; i < kStatsCh; ++i) s[i] = ss[i] = 0.0;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + t; e < total; e += stride) {
      const int64_t p = entries[e] >> 2;
      double4 m = make_double4(0.0, 0.0, 0.0, 0.0);
      if (c0 < 3) m = mu[entry_vertex[e]];
#pragma unroll
      for (int i = 0; i < kStatsCh; ++i) {
        const int c = c0 + i;
        if (c >= cin) break;
        float x;
        if (c == 0) x = row_coord(pos[3 * p], sc0, m.x);
        else if (c == 1) x = row_coord(pos[3 * p + 1], sc1, m.y);
        else if (c == 2) x = row_coord(pos[3 * p + 2], sc2, m.z);
        else x = feat[p * ld_feat + (c - 3)];
        s[i] += x;
        ss[i] += static_cast<double>(x) * x;
      }
    }
    double* o = part + static_cast<int64_t>(blockIdx.x) * 2 * cin;
    for (int i = 0; i < kStatsCh && c0 + i < cin; ++i) {
      __syncthreads();
      sh[0][t] = s[i];
      sh[1][t] = ss[i];
      __syncthreads();
      for (int off = kBlock / 2; off > 0; off >>= 1) {
        if (t < off) {
          sh[0][t] += sh[0][t + off];
          sh[1][t] += sh[1][t + off];
        }
        __syncthreads();
      }
      if (t == 0) {
        o[c0 + i] = sh[0][0];
        o[cin + c0 + i] = sh[1][0];
      }
    }
  }
}

// ---- the three [GN, ReLU, 1x1] blocks and the maximum over J_v ----
// A wave owns the list entries [r0, r0 + R) and walks them 64 at a time (one
// entry per lane for the gathers), then 16 at a time through the layers.
// The activations stay in registers: with A = weights (16 outputs x 4
// inputs) and B = activations transposed (4 inputs x 16 entries),
// v_mfma_f32_16x16x4_f32 leaves in lane (entry i, group g) the outputs
// 4g..4g+3 of entry i, which is the B operand of the next layer once that
// layer takes its inputs in the order (block b, register r): input
// 16b + 4g + r in lane group g.  The normalisation and ReLU of a layer's
// input are applied to those registers (per-channel scale and shift from
// LDS).  The weights sit in LDS in fragment order, one 64-float run per k
// step, so every A read is one conflict-free ds_read_b32.
// STAGE 1 and 2 stop after layer 1 / 2 and add up, in fp64, the values and
// squares of that layer's outputs over the rows (the next normalisation's
// statistics): per lane over its rows, then across the 16 row lanes of a
// lane group by a fixed butterfly, then over the waves in order into one
// partial per workgroup.  STAGE 3 runs all three layers and the maximum over
// J_v: a segmented scan across the 16 entry lanes (lists are contiguous and
// sorted by vertex); the segment still open at the end of 16 entries is
// carried into the next 16.  A list cut by a range boundary is finished with
// an order-independent atomic maximum on a row the mean pass set to -inf;
// every other list is stored.  If any normalisation parameter is not finite
// (a NaN or infinite input reached the statistics) every output is NaN.
constexpr int kWaves = kBlock / 64;
constexpr int kMaxBlocks = kMaxC / 16;
constexpr int kMaxK1Steps = kMaxC / 4;

constexpr int kTilePitch = 64 + 4;   // row pitch of a wave's 16 x 64 output tile
constexpr int kMlpRange = 128;       // list entries per wave of the MLP pass

struct MlpLds {
  size_t a1, a2, a3, b, g, x, o, end;   // in floats
  __host__ __device__ MlpLds(int ks1, int nb1, int nb2, int nb3) {
    a1 = 0;
    a2 = a1 + static_cast<size_t>(nb1) * ks1 * 64;
    a3 = a2 + static_cast<size_t>(nb2) * nb1 * 4 * 64;
    b = a3 + static_cast<size_t>(nb3) * nb2 * 4 * 64;
    g = b + 16 * static_cast<size_t>(nb1 + nb2 + nb3);
    x = g + 3 * static_cast<size_t>(kPreStride);   // normalisation tables of the three layer inputs
    o = x + static_cast<size_t>(kWaves) * 4 * ks1 * 64;   // per wave: 4 groups of 16 entries x ks1 k steps
    end = o + static_cast<size_t>(kWaves) * 16 * kTilePitch;
  }
  __host__ __device__ size_t bytes() const { return end * 4; }
};
static_assert(16 * kTilePitch * 4 >= 2 * kMaxC * 8, "a wave's output tile holds its statistics");

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// max into *a of the float with bits u, for any mix of signs: non-negative
// floats order like their bit patterns as signed integers, negative ones
// inversely as unsigned integers (a NaN with a clear sign bit, as written
// here, wins over every number)
__device__ inline void atomic_max_f32_bits(float* a, unsigned u) {
  if (u >> 31) atomicMin(reinterpret_cast<unsigned*>(a), u);
  else atomicMax(reinterpret_cast<int*>(a), static_cast<int>(u));
}

// Lane c holds output channel c of vertex v's maximum, or NaN when `bad`.
__device__ inline void emit_col(float* __restrict__ out, int64_t ld_out, int32_t v, bool shared, float m, bool bad,
                                int c3, int lane) {
  if (lane >= c3) return;
  const unsigned u = bad ? 0x7fc00000u : __float_as_uint(m);
  float* o = out + static_cast<int64_t>(v) * ld_out + lane;
  if (shared) atomic_max_f32_bits(o, u);
  else *reinterpret_cast<unsigned*>(o) = u;
}

// not finite (NaN or infinite), tested on the bits
__device__ inline bool nonfinite_bits(float x) {
  return (__float_as_uint(x) & 0x7f800000u) == 0x7f800000u;
}

// dst[q] = f(q) for q < count, BATCH independent loads in flight per thread
template <int BATCH, class F>
__device__ inline void stage(float* dst, int count, F f) {
  for (int q0 = threadIdx.x; q0 < count; q0 += BATCH * kBlock) {
    float v[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int q = q0 + j * kBlock;
      v[j] = q < count ? f(q) : 0.f;
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int q = q0 + j * kBlock;
      if (q < count) dst[q] = v[j];
    }
  }
}

// Fixed-count variant of stage(): the values are loaded into registers by
// load() and written to LDS by store(), so that other loads can be issued
// in between.
template <int COUNT>
struct Staged {
  static constexpr int N = (COUNT + kBlock - 1) / kBlock;
  float v[N];
  template <class F>
  __device__ void load(F f) {
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const int q = threadIdx.x + j * kBlock;
      v[j] = q < COUNT ? f(q) : 0.f;
    }
  }
  __device__ void store(float* dst) const {
#pragma unroll
    for (int j = 0; j < N; ++j) {
      const int q = threadIdx.x + j * kBlock;
      if (q < COUNT) dst[q] = v[j];
    }
  }
};

// Per-lane fp64 sums of a layer's outputs (channels 16 nb + 4 g + r of the
// lane's row) and of their squares.
template <int NB>
struct LayerStats {
  double s[NB][4], q[NB][4];
  __device__ LayerStats() {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) s[nb][r] = q[nb][r] = 0.0;
  }
  __device__ void add(const f32x4* h, bool valid) {
    if (!valid) return;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const double x = h[nb][r];
        s[nb][r] += x;
        q[nb][r] += x * x;
      }
  }
  // sums over the 16 row lanes of each lane group (xor butterfly), then
  // lane 16 g writes channels 16 nb + 4 g + r of its wave's column
  __device__ void to_lds(double* red, int lane) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          s[nb][r] += __shfl_xor(s[nb][r], off);
          q[nb][r] += __shfl_xor(q[nb][r], off);
        }
    if ((lane & 15) == 0) {
      const int g = lane >> 4;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          red[16 * nb + 4 * g + r] = s[nb][r];
          red[kMaxC + 16 * nb + 4 * g + r] = q[nb][r];
        }
    }
  }
};

// NB1..NB3: blocks of 16 outputs per layer; KS1: k steps of the first layer,
// or 0 for the runtime ks1.  Layers narrower than the instance run
// zero-padded (zero weights, biases and normalisation parameters: the padded
// hidden units are relu(0) = 0 and the padded outputs are not written).
// With KS1 > 0 the whole range's gathers and the weights are loaded into
// registers before the workgroup's first barrier, so their latencies
// overlap; with KS1 = 0 (any feature count) the rows are gathered into LDS
// 64 at a time.  WPE: waves per SIMD the register allocation must allow.
// pre: the three normalisation tables, kPreStride floats apart, each the C
// scales then the C shifts of its layer's input (C = 3 + cf, c1, c2).
// part (STAGE 1, 2): per workgroup the sums, then the sums of squares, of
// the c1 (STAGE 1) or c2 (STAGE 2) outputs.
template <int NB1, int NB2, int NB3, int KS1, int WPE, int STAGE>
__global__ void __launch_bounds__(kBlock, WPE)
k_dist_mlp(const int32_t* __restrict__ entries, const int32_t* __restrict__ entry_vertex, int64_t total,
           const float* __restrict__ pos, double sc0, double sc1, double sc2, const float* __restrict__ feat,
           int64_t ld_feat, int cf, const double4* __restrict__ mu, const float* __restrict__ pre,
           const float* __restrict__ W1, const float* __restrict__ b1, const float* __restrict__ W2,
           const float* __restrict__ b2, const float* __restrict__ W3, const float* __restrict__ b3, int ks1_rt,
           int c1, int c2, int c3, float* __restrict__ out, int64_t ld_out, double* __restrict__ part) {
  constexpr bool kPre = KS1 > 0;
  constexpr int kPer = kMlpRange / 64;   // groups of 64 entries per wave
  constexpr int NBS = STAGE == 1 ? NB1 : (STAGE == 2 ? NB2 : 1);
  extern __shared__ __align__(16) float sm[];
  const int ks1 = kPre ? KS1 : ks1_rt;
  const MlpLds lay(ks1, NB1, NB2, NB3);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int64_t r0 = (static_cast<int64_t>(blockIdx.x) * kWaves + wave) * kMlpRange;
  const bool active = r0 < total;
  const int64_t r1 = active ? min(r0 + kMlpRange, total) : r0;
  const int cin = 3 + cf;

  // weight fragments: run (nb, k step) holds, for lane (i, g), the weight of
  // output 16 nb + i and the k step's input for lane group g
  auto w1_at = [&](int q) {
    const int run = q >> 6, L = q & 63;
    const int nb = run / ks1, ks = run - nb * ks1;
    const int o = 16 * nb + (L & 15);
    const int k = 4 * ks + (L >> 4);   // 0..2 coordinates, 3 a zero pad, 4.. features
    const int src = k < 3 ? k : (k == 3 ? -1 : (k - 4 < cf ? k - 1 : -1));
    return (o < c1 && src >= 0) ? W1[o * cin + src] : 0.f;
  };
  // layers 2 and 3: the 4 k steps (kb, r = 0..3) of input block kb are
  // consecutive per lane, one ds_read_b128 per (nb, kb)
  auto w2_at = [&](int q) {
    const int r = q & 3, L = (q >> 2) & 63, run = q >> 8;
    const int nb = run / NB1, kb = run - nb * NB1;
    const int o = 16 * nb + (L & 15), k = 16 * kb + 4 * (L >> 4) + r;
    return (o < c2 && k < c1) ? W2[o * c1 + k] : 0.f;
  };
  auto w3_at = [&](int q) {
    const int r = q & 3, L = (q >> 2) & 63, run = q >> 8;
    const int nb = run / NB2, kb = run - nb * NB2;
    const int o = 16 * nb + (L & 15), k = 16 * kb + 4 * (L >> 4) + r;
    return (o < c3 && k < c2) ? W3[o * c2 + k] : 0.f;
  };
  auto b_at = [&](int i) {
    if (i < 16 * NB1) return (i < c1 && b1) ? b1[i] : 0.f;
    i -= 16 * NB1;
    if (i < 16 * NB2) return (i < c2 && b2) ? b2[i] : 0.f;
    i -= 16 * NB2;
    return (i < c3 && b3) ? b3[i] : 0.f;
  };
  // normalisation tables by input slot: table 0 indexed by the first layer's
  // k (k = 3 is the zero pad), tables 1 and 2 by channel; scales at [0, 64),
  // shifts at [64, 128) of each table
  auto g_at = [&](int q) {
    const int tab = q / kPreStride, w = q - tab * kPreStride;
    const int sh = w >= kMaxC, k = w - (sh ? kMaxC : 0);
    int ch, C;
    if (tab == 0) {
      ch = k < 3 ? k : (k == 3 ? -1 : (k - 4 < cf ? k - 1 : -1));
      C = cin;
    } else {
      C = tab == 1 ? c1 : c2;
      ch = k < C ? k : -1;
    }
    return ch >= 0 ? pre[tab * kPreStride + sh * C + ch] : 0.f;
  };
  // any parameter of the used normalisations that is not finite
  bool bad_local = false;
  if constexpr (STAGE == 3) {
    for (int q = t; q < 3 * kPreStride; q += kBlock) {
      const int tab = q / kPreStride, w = q - tab * kPreStride;
      const int C = tab == 0 ? cin : (tab == 1 ? c1 : c2);
      if ((w % kMaxC) < C && nonfinite_bits(pre[tab * kPreStride + (w >= kMaxC ? C : 0) + (w % kMaxC)]))
        bad_local = true;
    }
  }

  // per lane: vertex and input row [g / sigma - mu (fp64, rounded once), 0, f]
  // of entry r0 + 64 j + lane (registers only when kPre)
  constexpr int kRow = kPre ? 4 * KS1 : 1;
  int32_t vtx[kPer];
  float xr[kPre ? kPer : 1][kRow];
  int32_t key_before = -1, key_after = -1;   // the vertices whose lists run past the range's two ends
  if constexpr (kPre) {
    Staged<NB1 * KS1 * 64> s1;
    Staged<(STAGE >= 2 ? NB2 * NB1 * 4 * 64 : 1)> s2;
    Staged<(STAGE >= 3 ? NB3 * NB2 * 4 * 64 : 1)> s3;
    Staged<16 * (NB1 + NB2 + NB3)> sb;
    Staged<3 * kPreStride> sg;
    s1.load(w1_at);
    if constexpr (STAGE >= 2) s2.load(w2_at);
    if constexpr (STAGE >= 3) s3.load(w3_at);
    sb.load(b_at);
    sg.load(g_at);
    int32_t ent[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int64_t s = r0 + 64 * j + lane;
      ent[j] = s < r1 ? entries[s] : -1;
      vtx[j] = s < r1 ? entry_vertex[s] : -1;
    }
    key_before = (active && r0 > 0) ? entry_vertex[r0 - 1] : -1;
    key_after = (active && r1 < total) ? entry_vertex[r1] : -1;
    float g[kPer][3];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int64_t p = ent[j] >= 0 ? ent[j] >> 2 : 0;
#pragma unroll
      for (int c = 0; c < 3; ++c) g[j][c] = ent[j] >= 0 ? pos[3 * p + c] : 0.f;
      xr[j][3] = 0.f;
#pragma unroll
      for (int f = 0; f < kRow - 4; ++f) xr[j][4 + f] = (ent[j] >= 0 && f < cf) ? feat[p * ld_feat + f] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      double4 m = make_double4(0.0, 0.0, 0.0, 0.0);
      if (vtx[j] >= 0) m = mu[vtx[j]];
      xr[j][0] = row_coord(g[j][0], sc0, m.x);
      xr[j][1] = row_coord(g[j][1], sc1, m.y);
      xr[j][2] = row_coord(g[j][2], sc2, m.z);
    }
    s1.store(sm + lay.a1);
    if constexpr (STAGE >= 2) s2.store(sm + lay.a2);
    if constexpr (STAGE >= 3) s3.store(sm + lay.a3);
    sb.store(sm + lay.b);
    sg.store(sm + lay.g);
  } else {
    stage<8>(sm + lay.a1, NB1 * ks1 * 64, w1_at);
    if constexpr (STAGE >= 2) stage<8>(sm + lay.a2, NB2 * NB1 * 4 * 64, w2_at);
    if constexpr (STAGE >= 3) stage<8>(sm + lay.a3, NB3 * NB2 * 4 * 64, w3_at);
    stage<2>(sm + lay.b, 16 * (NB1 + NB2 + NB3), b_at);
    stage<2>(sm + lay.g, 3 * kPreStride, g_at);
    if (active) {
      key_before = r0 > 0 ? entry_vertex[r0 - 1] : -1;
      key_after = r1 < total ? entry_vertex[r1] : -1;
    }
  }
  const bool bad = __syncthreads_or(bad_local) != 0;
  if (STAGE == 3 && !active) return;

  const float* A1 = sm + lay.a1 + lane;
  const f32x4* A2 = reinterpret_cast<const f32x4*>(sm + lay.a2) + lane;
  const f32x4* A3 = reinterpret_cast<const f32x4*>(sm + lay.a3) + lane;
  const float* bias = sm + lay.b + 4 * lg;
  const float* G0 = sm + lay.g;                               // by first-layer k
  const float* G1 = sm + lay.g + kPreStride + 4 * lg;         // by channel 16 kb + 4 g + r
  const float* G2 = sm + lay.g + 2 * kPreStride + 4 * lg;
  float* X = sm + lay.x + static_cast<size_t>(wave) * 4 * ks1 * 64;
  float* T = sm + lay.o + static_cast<size_t>(wave) * 16 * kTilePitch;
  int32_t ckey = -1;   // vertex whose maximum is open (wave-uniform)
  float cmax = 0.f;    // its running maximum, channel `lane`
  LayerStats<NBS> stats;

#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int64_t base = r0 + 64 * j;
    if (base >= r1) break;
    // the 64 rows, normalised and rectified, as B fragments: group lane/16,
    // k step k/4, slot 16 (k%4) + lane%16
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // the last group's reads of X come first
    float* xs = X + (lane >> 4) * ks1 * 64 + (lane & 15);
    auto norm0 = [&](int k, float x) { return fmaxf(fmaf(x, G0[k], G0[kMaxC + k]), 0.f); };
    int32_t v;
    if constexpr (kPre) {
      v = vtx[j];
#pragma unroll
      for (int k = 0; k < kRow; ++k) xs[(k >> 2) * 64 + (k & 3) * 16] = v >= 0 ? norm0(k, xr[j][k]) : 0.f;
    } else {
      const int64_t s = base + lane;
      v = -1;
      if (s < r1) {
        const int32_t e = entries[s];
        v = entry_vertex[s];
        const int64_t p = e >> 2;
        const double4 m = mu[v];
        xs[0] = norm0(0, row_coord(pos[3 * p], sc0, m.x));
        xs[16] = norm0(1, row_coord(pos[3 * p + 1], sc1, m.y));
        xs[32] = norm0(2, row_coord(pos[3 * p + 2], sc2, m.z));
        xs[48] = 0.f;
        for (int k = 4; k < 4 * ks1; ++k)
          xs[(k >> 2) * 64 + (k & 3) * 16] = k - 4 < cf ? norm0(k, feat[p * ld_feat + (k - 4)]) : 0.f;
      } else {
        for (int k = 0; k < 4 * ks1; ++k) xs[(k >> 2) * 64 + (k & 3) * 16] = 0.f;
      }
    }
    // a wave's LDS accesses take effect in order; the fence keeps the
    // compiler from moving the reads above the writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    const int groups = static_cast<int>(min<int64_t>(4, (r1 - base + 15) / 16));
    for (int grp = 0; grp < groups; ++grp) {
      // weights and biases are read from LDS again for every 16 entries
      // (this compiler barrier stops them from being hoisted into registers
      // for the whole loop, which would cut the resident waves)
      __asm__ volatile("" ::: "memory");
      // (the shuffles run on all lanes: a lane masked off would read as 0)
      const int32_t krow = __shfl(v, 16 * grp + li);
      f32x4 h1[NB1], h2[NB2], o3[NB3];
#pragma unroll
      for (int nb = 0; nb < NB1; ++nb) h1[nb] = *reinterpret_cast<const f32x4*>(bias + 16 * nb);
      const float* xg = X + grp * ks1 * 64 + lane;
      if constexpr (kPre) {
#pragma unroll
        for (int ks = 0; ks < KS1; ++ks) {
          const float x = xg[ks * 64];
#pragma unroll
          for (int nb = 0; nb < NB1; ++nb) h1[nb] = mfma4(A1[(nb * KS1 + ks) * 64], x, h1[nb]);
        }
      } else {
        for (int ks = 0; ks < ks1; ++ks) {
          const float x = xg[ks * 64];
#pragma unroll
          for (int nb = 0; nb < NB1; ++nb) h1[nb] = mfma4(A1[(nb * ks1 + ks) * 64], x, h1[nb]);
        }
      }
      if constexpr (STAGE == 1) {
        stats.add(h1, krow >= 0);
        continue;
      }
#pragma unroll
      for (int nb = 0; nb < NB2; ++nb) h2[nb] = *reinterpret_cast<const f32x4*>(bias + 16 * NB1 + 16 * nb);
#pragma unroll
      for (int kb = 0; kb < NB1; ++kb) {
        f32x4 w[NB2];
#pragma unroll
        for (int nb = 0; nb < NB2; ++nb) w[nb] = A2[(nb * NB1 + kb) * 64];
        const f32x4 gs = *reinterpret_cast<const f32x4*>(G1 + 16 * kb);
        const f32x4 gt = *reinterpret_cast<const f32x4*>(G1 + kMaxC + 16 * kb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = fmaxf(fmaf(h1[kb][r], gs[r], gt[r]), 0.f);
#pragma unroll
          for (int nb = 0; nb < NB2; ++nb) h2[nb] = mfma4(w[nb][r], x, h2[nb]);
        }
      }
      if constexpr (STAGE == 2) {
        stats.add(h2, krow >= 0);
        continue;
      }
#pragma unroll
      for (int nb = 0; nb < NB3; ++nb)
        o3[nb] = *reinterpret_cast<const f32x4*>(bias + 16 * (NB1 + NB2) + 16 * nb);
#pragma unroll
      for (int kb = 0; kb < NB2; ++kb) {
        f32x4 w[NB3];
#pragma unroll
        for (int nb = 0; nb < NB3; ++nb) w[nb] = A3[(nb * NB2 + kb) * 64];
        const f32x4 gs = *reinterpret_cast<const f32x4*>(G2 + 16 * kb);
        const f32x4 gt = *reinterpret_cast<const f32x4*>(G2 + kMaxC + 16 * kb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = fmaxf(fmaf(h2[kb][r], gs[r], gt[r]), 0.f);
#pragma unroll
          for (int nb = 0; nb < NB3; ++nb) o3[nb] = mfma4(w[nb][r], x, o3[nb]);
        }
      }

      // the 16 x 64 outputs go through LDS; lane c then walks channel c
      // down the 16 rows.  Rows of one vertex are contiguous, so a row whose
      // vertex differs from the row before (bit i of the wave-uniform mask
      // `starts`) closes the open maximum.  Rows past the range carry
      // vertex -1, which is never written.
#pragma unroll
      for (int nb = 0; nb < NB3; ++nb) *reinterpret_cast<f32x4*>(T + li * kTilePitch + 16 * nb + 4 * lg) = o3[nb];
      const int32_t kup = __shfl(v, (16 * grp + li + 63) & 63);
      const int32_t kprev = li > 0 ? kup : ckey;
      const uint32_t starts = static_cast<uint32_t>(__ballot(krow != kprev)) & 0xffffu;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float x = T[i * kTilePitch + lane];
        if ((starts >> i) & 1u) {
          if (ckey >= 0)
            emit_col(out, ld_out, ckey, ckey == key_before || ckey == key_after, cmax, bad, c3, lane);
          ckey = __builtin_amdgcn_readlane(v, 16 * grp + i);
          cmax = x;
        } else {
          cmax = fmaxf(cmax, x);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // the walk's reads come before the next tile's writes
    }
  }
  if constexpr (STAGE == 3) {
    if (ckey >= 0)
      emit_col(out, ld_out, ckey, ckey == key_before || ckey == key_after, cmax, bad, c3, lane);
  } else {
    // the workgroup's partial: the waves' columns added in wave order
    double* red = reinterpret_cast<double*>(T);
    stats.to_lds(red, lane);
    __syncthreads();
    const int cst = STAGE == 1 ? c1 : c2;
    if (t < cst) {
      double a = 0.0, b = 0.0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const double* rw = reinterpret_cast<const double*>(sm + lay.o + static_cast<size_t>(w) * 16 * kTilePitch);
        a += rw[t];
        b += rw[kMaxC + t];
      }
      double* o = part + static_cast<int64_t>(blockIdx.x) * 2 * cst;
      o[t] = a;
      o[cst + t] = b;
    }
  }
}

// n x C rows of float32 (dense) to bfloat16 rows of stride ld, rounded to
// nearest even.
__global__ void __launch_bounds__(kBlock)
k_dist_to_bf16(const float* __restrict__ src, int64_t n, int C, uint16_t* __restrict__ dst, int64_t ld) {
  const int q4 = C / 4;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n * q4;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t v = i / q4;
    const int c = static_cast<int>(i - v * q4) * 4;
    const float4 x = *reinterpret_cast<const float4*>(src + v * C + c);
    *reinterpret_cast<uint2*>(dst + v * ld + c) = make_uint2(pack_bf16x2(x.x, x.y), pack_bf16x2(x.z, x.w));
  }
}

int64_t mlp_grid(int64_t total) {
  const int64_t waves = (total + kMlpRange - 1) / kMlpRange;
  return (waves + kWaves - 1) / kWaves;
}

template <int NB1, int NB2, int NB3, int KS1, int WPE>
void run_mlp(int stage, const MlpLds& lay, unsigned grid, hipStream_t s, const int32_t* entries, const int32_t* ev,
             int64_t total, const float* pos, const double sc[3], const float* feat, int64_t ld_feat, int cf,
             const double4* mu, const float* pre, const float* W1, const float* b1, const float* W2, const float* b2,
             const float* W3, const float* b3, int ks1, int C1, int C2, int C3, float* out, int64_t ld_out,
             double* part) {
  auto k1 = k_dist_mlp<NB1, NB2, NB3, KS1, WPE, 1>;
  auto k2 = k_dist_mlp<NB1, NB2, NB3, KS1, WPE, 2>;
  auto k3 = k_dist_mlp<NB1, NB2, NB3, KS1, WPE, 3>;
  auto kernel = stage == 1 ? k1 : (stage == 2 ? k2 : k3);
  if (!KS1) {
    // the runtime-width instance may need more than the default LDS limit
    static bool lds_limit_set[3] = {false, false, false};
    if (!lds_limit_set[stage - 1]) {
      const MlpLds worst(kMaxK1Steps, kMaxBlocks, kMaxBlocks, kMaxBlocks);
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(worst.bytes()));
      lds_limit_set[stage - 1] = true;
    }
  }
  launch(kernel, dim3(grid), dim3(kBlock), static_cast<uint32_t>(lay.bytes()), s, entries, ev, total, pos, sc[0],
         sc[1], sc[2], feat, ld_feat, cf, mu, pre, W1, b1, W2, b2, W3, b3, ks1, C1, C2, C3, out, ld_out, part);
}


// ---- Distribute + PointNet backward ----
// The forward is recomputed in fp64 with every block's input and
// activation kept (rows of list entries, in list order): the ReLU and the
// maximum are discrete decisions, and fp64 takes them as exact arithmetic
// does except within ~1e-15 of a tie.  The maximum routes dL/dx_v[c] to the
// row of J_v holding channel c's maximum (the first in list order); each
// block then goes backward in fp32 as a linear layer
// (launch_linear_backward, on the fp32 activations) and a GroupNorm + ReLU
// (launch_gn_backward, whose ReLU passes where the activation is > 0).  The
// raw rows are zero-padded to a multiple of 4 channels, each padding
// channel a group of its own that no weight reads.

// Raw rows (total x cin4) in fp64: g / sigma - mu, the features, zeros.
__global__ void __launch_bounds__(kBlock)
k_dist_raw_rows64(const int32_t* __restrict__ entries, const int32_t* __restrict__ entry_vertex, int64_t total,
                  const float* __restrict__ pos, double sc0, double sc1, double sc2, const double4* __restrict__ mu,
                  const float* __restrict__ feat, int64_t ld_feat, int cf, int cin4, double* __restrict__ H64) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (e >= total) return;
  const int64_t p = entries[e] >> 2;
  const double4 m = mu[entry_vertex[e]];
  double* r = H64 + e * cin4;
  r[0] = static_cast<double>(pos[3 * p]) / sc0 - m.x;
  r[1] = static_cast<double>(pos[3 * p + 1]) / sc1 - m.y;
  r[2] = static_cast<double>(pos[3 * p + 2]) / sc2 - m.z;
  for (int c = 0; c < cf; ++c) r[3 + c] = feat[p * ld_feat + c];
  for (int c = 3 + cf; c < cin4; ++c) r[c] = 0.0;
}

// Per-workgroup fp64 sums and sums of squares of each channel of fp64 rows
// [w rows_per, (w + 1) rows_per): thread t takes channel t % C of rows
// t / C, + slots, ...; the slots are added in order.  Layout as
// launch_gn_finalize reads it.
__global__ void __launch_bounds__(kBlock)
k_dist_stats64(const double* __restrict__ H, int C, int64_t n, int64_t rows_per, double* __restrict__ part) {
  __shared__ double sh[2][kBlock];
  const int t = threadIdx.x;
  const int slots = kBlock / C;
  const int c = t % C, slot = t / C;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rows_per;
  const int64_t r1 = min(r0 + rows_per, n);
  double s = 0.0, ss = 0.0;
  if (slot < slots)
    for (int64_t v = r0 + slot; v < r1; v += slots) {
      const double x = H[v * C + c];
      s += x;
      ss += x * x;
    }
  sh[0][t] = s;
  sh[1][t] = ss;
  __syncthreads();
  if (t < C) {
    double a = 0.0, b = 0.0;
    for (int sl = 0; sl < slots; ++sl) {
      a += sh[0][sl * C + t];
      b += sh[1][sl * C + t];
    }
    part[static_cast<int64_t>(blockIdx.x) * 2 * C + t] = a;
    part[static_cast<int64_t>(blockIdx.x) * 2 * C + C + t] = b;
  }
}

// One block forward in fp64 for every row:
//   xhat = (h - mean_g) inv_g,  a = max(xhat gamma_c + beta_c, 0),  h' = W a + b,
// writing xhat and a (fp32: what the backward of the block reads) and h'
// (fp64).  W (co x ci fp32, dense) is staged in LDS as fp64 rows of kMaxC,
// zero-padded; one thread per row.
__global__ void __launch_bounds__(kBlock)
k_dist_layer64(const double* __restrict__ Hin, int ci, const double* __restrict__ stats, int groups,
               const float* __restrict__ gamma, const float* __restrict__ beta, const float* __restrict__ W,
               const float* __restrict__ b, int co, int64_t rows, float* __restrict__ Xh32, float* __restrict__ A32,
               double* __restrict__ Hout) {
  __shared__ double sw[kMaxC * kMaxC];
  __shared__ double sb[kMaxC], smu[kMaxC], siv[kMaxC], sg[kMaxC], sbt[kMaxC];
  for (int i = threadIdx.x; i < co * kMaxC; i += kBlock) {
    const int o = i / kMaxC, c = i - o * kMaxC;
    sw[i] = c < ci ? static_cast<double>(W[o * ci + c]) : 0.0;
  }
  for (int i = threadIdx.x; i < co; i += kBlock) sb[i] = b ? b[i] : 0.0;
  const int per = ci / groups;
  for (int i = threadIdx.x; i < kMaxC; i += kBlock) {
    const bool in = i < ci;
    smu[i] = in ? stats[2 * (i / per)] : 0.0;
    siv[i] = in ? stats[2 * (i / per) + 1] : 0.0;
    sg[i] = in && gamma ? gamma[i] : 1.0;
    sbt[i] = in && beta ? beta[i] : 0.0;
  }
  __syncthreads();
  const int64_t r = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (r >= rows) return;
  double a[kMaxC];
#pragma unroll
  for (int i = 0; i < kMaxC; ++i) {
    const double x = i < ci ? Hin[r * ci + i] : 0.0;
    const double xh = (x - smu[i]) * siv[i];
    a[i] = i < ci ? fmax(xh * sg[i] + sbt[i], 0.0) : 0.0;
    if (i < ci) {
      Xh32[r * ci + i] = static_cast<float>(xh);
      A32[r * ci + i] = static_cast<float>(a[i]);
    }
  }
  for (int o = 0; o < co; ++o) {
    double v = sb[o];
#pragma unroll
    for (int i = 0; i < kMaxC; ++i) v = fma(sw[o * kMaxC + i], a[i], v);
    Hout[r * co + o] = v;
  }
}

// The maximum's gradient: thread (v, c) finds the first row of J_v holding
// channel c's maximum (fp64 rows) and writes dX[v][c] there (dH3 is zero
// elsewhere).
__global__ void __launch_bounds__(kBlock)
k_dist_route_max(const int32_t* __restrict__ offsets, int64_t n, const double* __restrict__ H3, int C3,
                 const float* __restrict__ dX, int64_t ld_dX, float* __restrict__ dH3) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n * C3) return;
  const int64_t v = i / C3;
  const int c = static_cast<int>(i - v * C3);
  const int64_t b = offsets[v], e = offsets[v + 1];
  if (b >= e) return;
  int64_t best = b;
  double top = H3[b * C3 + c];
  for (int64_t r = b + 1; r < e; ++r) {
    const double x = H3[r * C3 + c];
    if (x > top) {
      top = x;
      best = r;
    }
  }
  dH3[best * C3 + c] = dX[v * ld_dX + c];
}

__global__ void __launch_bounds__(kBlock)
k_dist_zero(float* __restrict__ x, int64_t count) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * kBlock)
    x[i] = 0.f;
}

// List position of every reference: at[entries[s]] = s.
__global__ void __launch_bounds__(kBlock)
k_dist_entry_at(const int32_t* __restrict__ entries, int64_t total, int32_t* __restrict__ at) {
  const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (s < total) at[entries[s]] = static_cast<int32_t>(s);
}

// dF_p[c] = sum over the d+1 rows of point p (vertex slots in order) of the
// feature part of dH0.
__global__ void __launch_bounds__(kBlock)
k_dist_dfeat(const int32_t* __restrict__ at, int64_t m, const float* __restrict__ dH0, int cin4, int cf,
             float* __restrict__ dF, int64_t ld_dF) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= m * cf) return;
  const int64_t p = i / cf;
  const int c = static_cast<int>(i - p * cf);
  float a = 0.f;
  for (int k = 0; k < 4; ++k) a += dH0[static_cast<int64_t>(at[4 * p + k]) * cin4 + 3 + c];
  dF[p * ld_dF + c] = a;
}

// Zero-padded copies of the first layer's weights (C1 x cin -> C1 x cin4)
// and of the raw rows' gamma / beta (padding: 1 / 0).
__global__ void __launch_bounds__(kBlock)
k_dist_pad_params(const float* __restrict__ W1, int C1, int cin, int cin4, const float* __restrict__ gamma,
                  const float* __restrict__ beta, float* __restrict__ W1p, float* __restrict__ gp,
                  float* __restrict__ bp) {
  for (int i = threadIdx.x; i < C1 * cin4; i += kBlock) {
    const int o = i / cin4, c = i - o * cin4;
    W1p[i] = c < cin ? W1[o * cin + c] : 0.f;
  }
  for (int c = threadIdx.x; c < cin4; c += kBlock) {
    gp[c] = c < cin && gamma ? gamma[c] : 1.f;
    bp[c] = c < cin && beta ? beta[c] : 0.f;
  }
}

// rows per workgroup of k_dist_stats64 and the number of workgroups
void stats64_parts(int64_t n, int C, int64_t* nparts, int64_t* rows_per) {
  const int slots = kBlock / C;
  int64_t rp = std::max<int64_t>(slots, (n + kStatsMaxParts - 1) / kStatsMaxParts);
  rp = (rp + slots - 1) / slots * slots;
  *rows_per = rp;
  *nparts = std::max<int64_t>(1, (n + rp - 1) / rp);
}

inline unsigned grid_rows(int64_t rows) {
  return static_cast<unsigned>(std::max<int64_t>(1, (rows + kBlock - 1) / kBlock));
}

}  // namespace

// Work space: the vertex means (n double4), the mean pass's span partials, the
// vertex of every list entry, the three normalisation tables, the
// statistics partials (at most max(512, MLP workgroups) x 2 x 64 doubles),
// and for a bfloat16 output the float32 rows (n x C3) it is rounded from.
int64_t distribute_workspace_bytes(int64_t n, int64_t total, int C3, int out_bf16) {
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  const int64_t parts = std::max<int64_t>(kStatsMaxParts, mlp_grid(total));
  auto up = [](int64_t b) { return (b + 255) / 256 * 256; };
  return up(32 * n) + up(2 * mean_spans * 32) + up(4 * total) + up(3 * kPreStride * 4) + up(parts * 2 * kMaxC * 8) +
         (out_bf16 ? up(4 * n * static_cast<int64_t>(C3)) : 0);
}

int distribute_max_features() { return kMaxIn - 3; }

void launch_distribute(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                       int64_t n, int64_t total, const float* pos, const double scale[3], const float* feat,
                       int64_t ld_feat, int cf, const float* gamma, const float* beta, float eps, const float* W1,
                       const float* b1, int C1, const float* W2, const float* b2, int C2, const float* W3,
                       const float* b3, int C3, void* out_dev, int out_bf16, int64_t ld_out_dev, void* work,
                       hipStream_t s) {
  if (total <= 0 || n <= 0) return;
  ScopedKernelTimer tm("distribute", s);
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  auto up = [](int64_t b) { return (b + 255) / 256 * 256; };
  char* w = static_cast<char*>(work);
  double4* mu4 = reinterpret_cast<double4*>(w);
  w += up(32 * n);
  double4* mh = reinterpret_cast<double4*>(w);
  double4* mt = mh + mean_spans;
  w += up(2 * mean_spans * 32);
  int32_t* ev = reinterpret_cast<int32_t*>(w);   // vertex of every list entry
  w += up(4 * total);
  float* pre = reinterpret_cast<float*>(w);
  w += up(3 * kPreStride * 4);
  double* part = reinterpret_cast<double*>(w);
  w += up(std::max<int64_t>(kStatsMaxParts, mlp_grid(total)) * 2 * kMaxC * 8);
  // the maxima are taken in float32: into the caller's rows, or into dense
  // work rows that are rounded to bfloat16 at the end
  float* out = out_bf16 ? reinterpret_cast<float*>(w) : static_cast<float*>(out_dev);
  const int64_t ld_out = out_bf16 ? C3 : ld_out_dev;
  launch(k_dist_mean, dim3(static_cast<unsigned>(mean_spans)), dim3(kBlock), 0, s, offsets, entries, chunk_first,
         chunk, n, total, pos, scale[0], scale[1], scale[2], mu4, mh, mt, ev, static_cast<int64_t>(kMlpRange), out,
         ld_out, C3);
  if (mean_spans > 1)
    launch(k_dist_mean_finish, dim3(static_cast<unsigned>((mean_spans + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
           offsets, chunk_first, chunk, mean_spans, mu4, static_cast<const double4*>(mh),
           static_cast<const double4*>(mt));
  // the raw rows' statistics -> table 0
  const int cin = 3 + cf;
  const int64_t np0 = std::min<int64_t>(kStatsMaxParts, (total + kBlock - 1) / kBlock);
  launch(k_dist_in_stats, dim3(static_cast<unsigned>(np0)), dim3(kBlock), 0, s, entries,
         static_cast<const int32_t*>(ev), total, pos, scale[0], scale[1], scale[2], static_cast<const double4*>(mu4),
         feat, ld_feat, cin, part);
  auto groups = [](int C) { return C <= 32 ? C : 32; };
  launch_gn_finalize(part, np0, cin, groups(cin), total, gamma, beta, eps, pre, s);

  const int ks1 = (4 + cf + 3) / 4;   // coordinates, a zero pad, features, in k steps of 4
  // the paper's 16-32-64 block (up to 4 raw features) has its own instance;
  // every other shape runs zero-padded to 64-64-64
  const bool paper = C1 == 16 && C2 == 32 && C3 == 64 && ks1 <= 2;
  const MlpLds lay = paper ? MlpLds(2, 1, 2, 4) : MlpLds(ks1, kMaxBlocks, kMaxBlocks, kMaxBlocks);
  const unsigned grid = static_cast<unsigned>(mlp_grid(total));
  const int64_t offs[3] = {0, cin, static_cast<int64_t>(cin) + C1};
  for (int stage = 1; stage <= 3; ++stage) {
    if (paper)
      run_mlp<1, 2, 4, 2, 4>(stage, lay, grid, s, entries, ev, total, pos, scale, feat, ld_feat, cf, mu4, pre, W1,
                             b1, W2, b2, W3, b3, ks1, C1, C2, C3, out, ld_out, part);
    else
      run_mlp<kMaxBlocks, kMaxBlocks, kMaxBlocks, 0, 1>(stage, lay, grid, s, entries, ev, total, pos, scale, feat,
                                                        ld_feat, cf, mu4, pre, W1, b1, W2, b2, W3, b3, ks1, C1, C2,
                                                        C3, out, ld_out, part);
    if (stage < 3) {
      const int C = stage == 1 ? C1 : C2;
      launch_gn_finalize(part, grid, C, groups(C), total, gamma ? gamma + offs[stage] : nullptr,
                         beta ? beta + offs[stage] : nullptr, eps, pre + stage * kPreStride, s);
    }
  }
  if (out_bf16)
    launch(k_dist_to_bf16, dim3(static_cast<unsigned>(std::min<int64_t>((n * C3 / 4 + kBlock - 1) / kBlock, 4096))),
           dim3(kBlock), 0, s, static_cast<const float*>(out), n, C3, static_cast<uint16_t*>(out_dev), ld_out_dev);
}

}  // namespace lat

namespace lat {

// Work space of the backward, carved in this order (each piece 256-byte
// aligned): means, mean partials, entry vertices, list positions, two fp64
// row buffers, the blocks' normalised inputs and activations (fp32), dH3, two gradient
// buffers, padded parameters, normalisation tables, stats, coefficients,
// statistics partials, linear-layer partials.
int64_t distribute_backward_workspace_bytes(int64_t n, int64_t m, int64_t total, int cf, int C1, int C2, int C3) {
  auto up = [](int64_t b) { return (b + 255) / 256 * 256; };
  const int cin4 = (3 + cf + 3) / 4 * 4;
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  const int64_t widest = std::max<int64_t>(std::max(cin4, C1), std::max(C2, C3));
  int64_t b = up(32 * n) + up(2 * mean_spans * 32) + up(4 * total) + up(4 * std::max<int64_t>(4 * m, 1));
  b += 2 * up(8 * total * widest);
  b += 2 * (up(4 * total * cin4) + up(4 * total * C1) + up(4 * total * C2));
  b += up(4 * total * C3) + 2 * up(4 * total * widest);
  b += up(4 * (C1 * cin4 + 2 * cin4 + 2 * cin4));
  b += 3 * up(4 * 2 * widest) + 3 * up(8 * 2 * widest) + up(4 * 4 * widest);
  // k_dist_stats64 runs at most kStatsMaxParts workgroups
  b += up(std::max<int64_t>(gn_workspace_bytes(total, static_cast<int>(widest)), kStatsMaxParts * 2 * widest * 8));
  int64_t lin = 0;
  const int ks[3] = {C1, C2, C3}, cs[3] = {cin4, C1, C2};
  for (int i = 0; i < 3; ++i) lin = std::max(lin, classify_backward_partial_floats(total, ks[i], cs[i]));
  b += up(4 * lin);
  return b;
}

void launch_distribute_backward(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                                int64_t n, int64_t m, int64_t total, const float* pos, const double scale[3],
                                const float* feat, int64_t ld_feat, int cf, const float* gamma, const float* beta,
                                float eps, const float* W1, const float* b1, int C1, const float* W2, const float* b2,
                                int C2, const float* W3, const float* b3, int C3, const float* dX, int64_t ld_dX,
                                float* dF, int64_t ld_dF, float* dW1, float* db1, float* dW2, float* db2, float* dW3,
                                float* db3, float* dgamma, float* dbeta, void* work, hipStream_t s) {
  ScopedKernelTimer tm("distribute_bwd", s);
  auto up = [](int64_t b) { return (b + 255) / 256 * 256; };
  const int cin = 3 + cf, cin4 = (cin + 3) / 4 * 4;
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  const int64_t widest = std::max<int64_t>(std::max(cin4, C1), std::max(C2, C3));
  char* w = static_cast<char*>(work);
  auto take = [&](int64_t bytes) {
    char* p = w;
    w += up(bytes);
    return p;
  };
  double4* mu4 = reinterpret_cast<double4*>(take(32 * n));
  double4* mh = reinterpret_cast<double4*>(take(2 * mean_spans * 32));
  double4* mt = mh + mean_spans;
  int32_t* ev = reinterpret_cast<int32_t*>(take(4 * total));
  int32_t* at = reinterpret_cast<int32_t*>(take(4 * std::max<int64_t>(4 * m, 1)));
  double* h64[2] = {reinterpret_cast<double*>(take(8 * total * widest)),
                    reinterpret_cast<double*>(take(8 * total * widest))};
  const int ci[3] = {cin4, C1, C2}, co[3] = {C1, C2, C3};
  float* Xh32[3];   // each block's normalised input
  float* A32[3];    // and its activation
  for (int i = 0; i < 3; ++i) Xh32[i] = reinterpret_cast<float*>(take(4 * total * ci[i]));
  for (int i = 0; i < 3; ++i) A32[i] = reinterpret_cast<float*>(take(4 * total * ci[i]));
  float* dH3 = reinterpret_cast<float*>(take(4 * total * C3));
  float* gA = reinterpret_cast<float*>(take(4 * total * widest));
  float* gB = reinterpret_cast<float*>(take(4 * total * widest));
  float* W1p = reinterpret_cast<float*>(take(4 * (C1 * cin4 + 2 * cin4 + 2 * cin4)));
  float* g0p = W1p + C1 * cin4;
  float* b0p = g0p + cin4;
  float* dg0 = b0p + cin4;
  float* db0 = dg0 + cin4;
  float* pre[3];
  double* stats[3];
  for (int i = 0; i < 3; ++i) pre[i] = reinterpret_cast<float*>(take(4 * 2 * widest));
  for (int i = 0; i < 3; ++i) stats[i] = reinterpret_cast<double*>(take(8 * 2 * widest));
  float* coef = reinterpret_cast<float*>(take(4 * 4 * widest));
  void* gnw = take(std::max<int64_t>(gn_workspace_bytes(total, static_cast<int>(widest)), kStatsMaxParts * 2 * widest * 8));
  float* part = reinterpret_cast<float*>(w);

  auto groups = [](int C) { return C <= 32 ? C : 32; };
  const float* gam[3] = {g0p, gamma ? gamma + cin : nullptr, gamma ? gamma + cin + C1 : nullptr};
  const float* bet[3] = {b0p, beta ? beta + cin : nullptr, beta ? beta + cin + C1 : nullptr};
  const float* Ws[3] = {W1p, W2, W3};
  const float* bs[3] = {b1, b2, b3};
  float* dWs[3] = {dW1, dW2, dW3};
  float* dbs[3] = {db1, db2, db3};
  const int wout[3] = {cin, C1, C2};
  float* dgam[3] = {dg0, dgamma ? dgamma + cin : nullptr, dgamma ? dgamma + cin + C1 : nullptr};
  float* dbet[3] = {db0, dbeta ? dbeta + cin : nullptr, dbeta ? dbeta + cin + C1 : nullptr};

  // forward in fp64, keeping every block's input and activation
  launch(k_dist_pad_params, dim3(1), dim3(kBlock), 0, s, W1, C1, cin, cin4, gamma, beta, W1p, g0p, b0p);
  if (total > 0) {
    launch(k_dist_mean, dim3(static_cast<unsigned>(mean_spans)), dim3(kBlock), 0, s, offsets, entries, chunk_first,
           chunk, n, total, pos, scale[0], scale[1], scale[2], mu4, mh, mt, ev, INT64_MAX, static_cast<float*>(nullptr),
           static_cast<int64_t>(0), 0);
    if (mean_spans > 1)
      launch(k_dist_mean_finish, dim3(static_cast<unsigned>((mean_spans + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
             offsets, chunk_first, chunk, mean_spans, mu4, static_cast<const double4*>(mh),
             static_cast<const double4*>(mt));
    launch(k_dist_raw_rows64, dim3(grid_rows(total)), dim3(kBlock), 0, s, entries, static_cast<const int32_t*>(ev),
           total, pos, scale[0], scale[1], scale[2], static_cast<const double4*>(mu4), feat, ld_feat, cf, cin4, h64[0]);
  }
  for (int i = 0; i < 3; ++i) {
    int64_t np, rp;
    stats64_parts(total, ci[i], &np, &rp);
    double* gpart = static_cast<double*>(gnw);
    if (total > 0)
      launch(k_dist_stats64, dim3(static_cast<unsigned>(np)), dim3(kBlock), 0, s, static_cast<const double*>(h64[i & 1]),
             ci[i], total, rp, gpart);
    launch_gn_finalize(gpart, np, ci[i], groups(ci[i]), total, gam[i], bet[i], eps, pre[i], s, stats[i]);
    if (total > 0)
      launch(k_dist_layer64, dim3(grid_rows(total)), dim3(kBlock), 0, s, static_cast<const double*>(h64[i & 1]), ci[i],
             static_cast<const double*>(stats[i]), groups(ci[i]), gam[i], bet[i], Ws[i], bs[i], co[i], total, Xh32[i],
             A32[i], h64[(i + 1) & 1]);
  }
  // the maximum, then the three blocks backward in fp32
  const unsigned zg = static_cast<unsigned>(std::min<int64_t>(8192, (total * C3 + kBlock - 1) / kBlock + 1));
  launch(k_dist_zero, dim3(zg), dim3(kBlock), 0, s, dH3, total * C3);
  if (n > 0)
    launch(k_dist_route_max, dim3(grid_rows(n * C3)), dim3(kBlock), 0, s, offsets, n,
           static_cast<const double*>(h64[1]), C3, dX, ld_dX, dH3);
  const float* g = dH3;
  for (int i = 2; i >= 0; --i) {
    // dA = g W_i, dW_i, db_i on the activations; then dH_i = GroupNorm +
    // ReLU backward of dA
    launch_linear_backward(g, co[i], Ws[i], co[i], ci[i], total, A32[i], ci[i], nullptr, gA, ci[i], dWs[i], wout[i],
                           dbs[i], part, s);
    launch_gn_backward(Xh32[i], ci[i], gA, ci[i], ci[i], groups(ci[i]), total, gam[i], nullptr, stats[i], dgam[i],
                       dbet[i], coef, gB, ci[i], gnw, s, A32[i], ci[i], true);
    g = gB;   // read by the next block's linear backward, which writes gA again
  }
  // g now holds dH0 (total x cin4)
  if (dgamma) (void)hipMemcpyAsync(dgamma, dg0, sizeof(float) * cin, hipMemcpyDeviceToDevice, s);
  if (dbeta) (void)hipMemcpyAsync(dbeta, db0, sizeof(float) * cin, hipMemcpyDeviceToDevice, s);
  if (dF && cf > 0 && m > 0) {
    launch(k_dist_entry_at, dim3(grid_rows(total)), dim3(kBlock), 0, s, entries, total, at);
    launch(k_dist_dfeat, dim3(grid_rows(m * cf)), dim3(kBlock), 0, s, static_cast<const int32_t*>(at), m, g, cin4,
           cf, dF, ld_dF);
  }
}

}  // namespace lat

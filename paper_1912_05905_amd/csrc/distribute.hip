// Distribute + PointNet on gfx950 (Proposed Operations, Eq. (distribute),
// and the PointNet block of the architecture figure):
//   x_v = max_{p in J_v} W3 relu(W2 relu(W1 [g_p - mu_v ; f_p] + b1) + b2) + b3,
//   mu_v = mean of g_p over J_v.
// J_v are the vertex lists built with the lattice (entries grouped by vertex).
// The mean runs over spans of 256 consecutive list entries, so the work is
// balanced however skewed the list lengths are: a vertex inside a span is
// finished there; the vertex a span starts inside and the vertex that runs
// past its end leave a head and a tail partial, which a finishing pass joins
// in span order.  The mean is summed in fp64 (positions can be tens of
// metres from the origin while g - mu is a fraction of sigma) and g - mu is
// rounded to fp32 once.  The three 1x1 layers run on
// v_mfma_f32_16x16x4_f32 with the activations held in registers; each wave
// takes an equal range of list entries and reduces the maximum across lanes.
#include <algorithm>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int kMeanSpan = kBlock;  // list entries per workgroup of the mean pass
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
            double4* __restrict__ part_tail, int32_t* __restrict__ entry_vertex, int64_t R,
            float* __restrict__ out, int64_t ld_out, int C3) {
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

// ---- the three 1x1 layers and the maximum over J_v ----
// A wave owns the list entries [r0, r0 + R) and walks them 64 at a time (one
// entry per lane for the gathers), then 16 at a time through the layers.
// The activations stay in registers: with A = weights (16 outputs x 4
// inputs) and B = activations transposed (4 inputs x 16 entries),
// v_mfma_f32_16x16x4_f32 leaves in lane (entry i, group g) the outputs
// 4g..4g+3 of entry i, which is the B operand of the next layer once that
// layer takes its inputs in the order (block b, register r): input
// 16b + 4g + r in lane group g.  The weights sit in LDS in that fragment
// order, one 64-float run per k step, so every A read is one conflict-free
// ds_read_b32.  The maximum over J_v is a segmented scan across the 16
// entry lanes (lists are contiguous and sorted by vertex); the segment
// still open at the end of 16 entries is carried into the next 16.  A list
// cut by a range boundary is finished with an order-independent atomic
// maximum on a row the mean pass set to -inf; every other list is stored.
constexpr int kWaves = kBlock / 64;
constexpr int kMaxBlocks = kMaxC / 16;
constexpr int kMaxK1Steps = kMaxC / 4;

constexpr int kTilePitch = 64 + 4;
constexpr int kMlpRange = 128;       // list entries per wave of the MLP pass   // row pitch of a wave's 16 x 64 output tile

struct MlpLds {
  size_t a1, a2, a3, b, x, o, end;   // in floats
  __host__ __device__ MlpLds(int ks1, int nb1, int nb2, int nb3) {
    a1 = 0;
    a2 = a1 + static_cast<size_t>(nb1) * ks1 * 64;
    a3 = a2 + static_cast<size_t>(nb2) * nb1 * 4 * 64;
    b = a3 + static_cast<size_t>(nb3) * nb2 * 4 * 64;
    x = b + 16 * static_cast<size_t>(nb1 + nb2 + nb3);
    o = x + static_cast<size_t>(kWaves) * 4 * ks1 * 64;   // per wave: 4 groups of 16 entries x ks1 k steps
    end = o + static_cast<size_t>(kWaves) * 16 * kTilePitch;
  }
  __host__ __device__ size_t bytes() const { return end * 4; }
};

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// max into *a for any mix of signs: non-negative floats order like their bit
// patterns as signed integers, negative ones inversely as unsigned integers
__device__ inline void atomic_max_f32(float* a, float x) {
  const unsigned u = __float_as_uint(x);
  if (u >> 31) atomicMin(reinterpret_cast<unsigned*>(a), u);
  else atomicMax(reinterpret_cast<int*>(a), static_cast<int>(u));
}

// Lane c holds output channel c of vertex v's maximum.
__device__ inline void emit_col(float* __restrict__ out, int64_t ld_out, int32_t v, bool shared, float m, int c3,
                                int lane) {
  if (lane >= c3) return;
  float* o = out + static_cast<int64_t>(v) * ld_out + lane;
  if (shared) atomic_max_f32(o, m);
  else *o = m;
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

// NB1..NB3: blocks of 16 outputs per layer; KS1: k steps of the first layer,
// or 0 for the runtime ks1.  Layers narrower than the instance run
// zero-padded (zero weights and biases: the padded hidden units are
// relu(0) = 0 and the padded outputs are not written).  With KS1 > 0 the
// whole range's gathers and the weights are loaded into registers before
// the workgroup's first barrier, so their latencies overlap; with KS1 = 0
// (any feature count) the rows are gathered into LDS 64 at a time.  WPE:
// waves per SIMD the register allocation must allow.
template <int NB1, int NB2, int NB3, int KS1, int WPE>
__global__ void __launch_bounds__(kBlock, WPE)
k_dist_mlp(const int32_t* __restrict__ entries, const int32_t* __restrict__ entry_vertex, int64_t total,
           const float* __restrict__ pos, const float* __restrict__ feat, int64_t ld_feat, int cf,
           const double4* __restrict__ mu, const float* __restrict__ W1, const float* __restrict__ b1,
           const float* __restrict__ W2, const float* __restrict__ b2, const float* __restrict__ W3,
           const float* __restrict__ b3, int ks1_rt, int c1, int c2, int c3, float* __restrict__ out,
           int64_t ld_out) {
  constexpr bool kPre = KS1 > 0;
  constexpr int kPer = kMlpRange / 64;   // groups of 64 entries per wave
  extern __shared__ __align__(16) float sm[];
  const int ks1 = kPre ? KS1 : ks1_rt;
  const MlpLds lay(ks1, NB1, NB2, NB3);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int64_t r0 = (static_cast<int64_t>(blockIdx.x) * kWaves + wave) * kMlpRange;
  const bool active = r0 < total;
  const int64_t r1 = active ? min(r0 + kMlpRange, total) : r0;

  // weight fragments: run (nb, k step) holds, for lane (i, g), the weight of
  // output 16 nb + i and the k step's input for lane group g
  const int cin = 3 + cf;
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

  // per lane: vertex and input row [g - mu (fp64, rounded once), 0, f] of
  // entry r0 + 64 j + lane (registers only when kPre)
  constexpr int kRow = kPre ? 4 * KS1 : 1;
  int32_t vtx[kPer];
  float xr[kPre ? kPer : 1][kRow];
  int32_t key_before = -1, key_after = -1;   // the vertices whose lists run past the range's two ends
  if constexpr (kPre) {
    Staged<NB1 * KS1 * 64> s1;
    Staged<NB2 * NB1 * 4 * 64> s2;
    Staged<NB3 * NB2 * 4 * 64> s3;
    Staged<16 * (NB1 + NB2 + NB3)> sb;
    s1.load(w1_at);
    s2.load(w2_at);
    s3.load(w3_at);
    sb.load(b_at);
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
      xr[j][0] = static_cast<float>(static_cast<double>(g[j][0]) - m.x);
      xr[j][1] = static_cast<float>(static_cast<double>(g[j][1]) - m.y);
      xr[j][2] = static_cast<float>(static_cast<double>(g[j][2]) - m.z);
    }
    s1.store(sm + lay.a1);
    s2.store(sm + lay.a2);
    s3.store(sm + lay.a3);
    sb.store(sm + lay.b);
  } else {
    stage<8>(sm + lay.a1, NB1 * ks1 * 64, w1_at);
    stage<8>(sm + lay.a2, NB2 * NB1 * 4 * 64, w2_at);
    stage<8>(sm + lay.a3, NB3 * NB2 * 4 * 64, w3_at);
    stage<2>(sm + lay.b, 16 * (NB1 + NB2 + NB3), b_at);
    if (active) {
      key_before = r0 > 0 ? entry_vertex[r0 - 1] : -1;
      key_after = r1 < total ? entry_vertex[r1] : -1;
    }
  }
  __syncthreads();
  if (!active) return;

  const float* A1 = sm + lay.a1 + lane;
  const f32x4* A2 = reinterpret_cast<const f32x4*>(sm + lay.a2) + lane;
  const f32x4* A3 = reinterpret_cast<const f32x4*>(sm + lay.a3) + lane;
  const float* bias = sm + lay.b + 4 * lg;
  float* X = sm + lay.x + static_cast<size_t>(wave) * 4 * ks1 * 64;
  float* T = sm + lay.o + static_cast<size_t>(wave) * 16 * kTilePitch;
  int32_t ckey = -1;   // vertex whose maximum is open (wave-uniform)
  float cmax = 0.f;    // its running maximum, channel `lane`

#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int64_t base = r0 + 64 * j;
    if (base >= r1) break;
    // the 64 rows as B fragments: group lane/16, k step k/4, slot
    // 16 (k%4) + lane%16
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // the last group's reads of X come first
    float* xs = X + (lane >> 4) * ks1 * 64 + (lane & 15);
    int32_t v;
    if constexpr (kPre) {
      v = vtx[j];
#pragma unroll
      for (int k = 0; k < kRow; ++k) xs[(k >> 2) * 64 + (k & 3) * 16] = xr[j][k];
    } else {
      const int64_t s = base + lane;
      v = -1;
      if (s < r1) {
        const int32_t e = entries[s];
        v = entry_vertex[s];
        const int64_t p = e >> 2;
        const double4 m = mu[v];
        xs[0] = static_cast<float>(static_cast<double>(pos[3 * p]) - m.x);
        xs[16] = static_cast<float>(static_cast<double>(pos[3 * p + 1]) - m.y);
        xs[32] = static_cast<float>(static_cast<double>(pos[3 * p + 2]) - m.z);
        xs[48] = 0.f;
        for (int k = 4; k < 4 * ks1; ++k)
          xs[(k >> 2) * 64 + (k & 3) * 16] = k - 4 < cf ? feat[p * ld_feat + (k - 4)] : 0.f;
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
#pragma unroll
      for (int nb = 0; nb < NB2; ++nb) h2[nb] = *reinterpret_cast<const f32x4*>(bias + 16 * NB1 + 16 * nb);
#pragma unroll
      for (int kb = 0; kb < NB1; ++kb) {
        f32x4 w[NB2];
#pragma unroll
        for (int nb = 0; nb < NB2; ++nb) w[nb] = A2[(nb * NB1 + kb) * 64];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = fmaxf(h1[kb][r], 0.f);
#pragma unroll
          for (int nb = 0; nb < NB2; ++nb) h2[nb] = mfma4(w[nb][r], x, h2[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB3; ++nb)
        o3[nb] = *reinterpret_cast<const f32x4*>(bias + 16 * (NB1 + NB2) + 16 * nb);
#pragma unroll
      for (int kb = 0; kb < NB2; ++kb) {
        f32x4 w[NB3];
#pragma unroll
        for (int nb = 0; nb < NB3; ++nb) w[nb] = A3[(nb * NB2 + kb) * 64];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = fmaxf(h2[kb][r], 0.f);
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
      // (both shuffles run on all lanes: a lane masked off would read as 0)
      const int32_t krow = __shfl(v, 16 * grp + li);
      const int32_t kup = __shfl(v, (16 * grp + li + 63) & 63);
      const int32_t kprev = li > 0 ? kup : ckey;
      const uint32_t starts = static_cast<uint32_t>(__ballot(krow != kprev)) & 0xffffu;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float x = T[i * kTilePitch + lane];
        if ((starts >> i) & 1u) {
          if (ckey >= 0) emit_col(out, ld_out, ckey, ckey == key_before || ckey == key_after, cmax, c3, lane);
          ckey = __builtin_amdgcn_readlane(v, 16 * grp + i);
          cmax = x;
        } else {
          cmax = fmaxf(cmax, x);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // the walk's reads come before the next tile's writes
    }
  }
  if (ckey >= 0) emit_col(out, ld_out, ckey, ckey == key_before || ckey == key_after, cmax, c3, lane);
}


}  // namespace

int64_t distribute_workspace_bytes(int64_t total, int C3) {
  (void)C3;
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  return 2 * mean_spans * static_cast<int64_t>(sizeof(double4)) + 4 * total;
}

int distribute_max_features() { return kMaxC - 4; }

void launch_distribute(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                       int64_t n, int64_t total, const float* pos, const float* feat, int64_t ld_feat, int cf,
                       const float* W1, const float* b1, int C1, const float* W2, const float* b2, int C2,
                       const float* W3, const float* b3, int C3, float* out, int64_t ld_out, double* mu, void* work,
                       hipStream_t s) {
  if (total <= 0 || n <= 0) return;
  ScopedKernelTimer tm("distribute", s);
  const int64_t mean_spans = (total + kMeanSpan - 1) / kMeanSpan;
  double4* mh = static_cast<double4*>(work);
  double4* mt = mh + mean_spans;
  int32_t* ev = reinterpret_cast<int32_t*>(mt + mean_spans);   // vertex of every list entry
  double4* mu4 = reinterpret_cast<double4*>(mu);
  launch(k_dist_mean, dim3(static_cast<unsigned>(mean_spans)), dim3(kBlock), 0, s, offsets, entries, chunk_first,
         chunk, n, total, pos, mu4, mh, mt, ev, static_cast<int64_t>(kMlpRange), out, ld_out, C3);
  if (mean_spans > 1)
    launch(k_dist_mean_finish, dim3(static_cast<unsigned>((mean_spans + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
           offsets, chunk_first, chunk, mean_spans, mu4, static_cast<const double4*>(mh),
           static_cast<const double4*>(mt));
  const int ks1 = (4 + cf + 3) / 4;   // coordinates, a zero pad, features, in k steps of 4
  // the paper's 16-32-64 block (up to 4 raw features) has its own instance;
  // every other shape runs zero-padded to 64-64-64
  const bool paper = C1 == 16 && C2 == 32 && C3 == 64 && ks1 <= 2;
  auto kernel = paper ? k_dist_mlp<1, 2, 4, 2, 4> : k_dist_mlp<kMaxBlocks, kMaxBlocks, kMaxBlocks, 0, 1>;
  const MlpLds lay = paper ? MlpLds(2, 1, 2, 4) : MlpLds(ks1, kMaxBlocks, kMaxBlocks, kMaxBlocks);
  static bool lds_limit_set = false;
  if (!lds_limit_set) {
    const MlpLds worst(kMaxK1Steps, kMaxBlocks, kMaxBlocks, kMaxBlocks);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_dist_mlp<kMaxBlocks, kMaxBlocks, kMaxBlocks, 0, 1>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(worst.bytes()));
    lds_limit_set = true;
  }
  const int64_t waves = (total + kMlpRange - 1) / kMlpRange;
  const unsigned grid = static_cast<unsigned>((waves + kWaves - 1) / kWaves);
  launch(kernel, dim3(grid), dim3(kBlock), static_cast<uint32_t>(lay.bytes()), s, entries,
         static_cast<const int32_t*>(ev), total, pos, feat, ld_feat, cf, static_cast<const double4*>(mu4), W1, b1, W2, b2, W3, b3, ks1, C1, C2, C3, out, ld_out);
}

}  // namespace lat

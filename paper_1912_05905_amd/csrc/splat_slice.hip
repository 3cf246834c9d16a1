// Splat, Slice and DeformSlice on gfx950.  All three are gathers bounded by
// HBM bandwidth: a row of C channels is handled by a group of LPR lanes
// (LPR a power of two), each lane moving 16 bytes (4 fp32 or 8 bf16 channels)
// per access so that a row is one contiguous, fully used transaction.
#include <algorithm>

#include <type_traits>
#include <utility>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int64_t kDeformBwdGrid = 1024;   // workgroups of the DeformSlice backward's per-point pass
constexpr unsigned kClassifyGrid = 2048;   // workgroups of the fused classifier (a multiple of 8)
constexpr int kClassifyMaxWeights = 16384; // K x C classifier weights staged in LDS

// float -> bfloat16, round to nearest even (NaN stays NaN).
// Row / chunk index of a lane group with XCD-contiguous workgroup order:
// workgroup b runs on XCD b % 8, so consecutive work items (which share
// feature or vertex rows) are given to workgroups of the same XCD and meet in
// its L2.  Launches use xcd_grid() workgroups.
template <int LPR>
__device__ inline int64_t xcd_item(unsigned nblocks_logical) {
  const unsigned b = blockIdx.x;
  const unsigned per = (nblocks_logical + 7) / 8;
  const int64_t logical = static_cast<int64_t>(b % 8) * per + b / 8;
  return (logical * kBlock + threadIdx.x) / LPR;
}

inline unsigned xcd_grid(unsigned nblocks_logical) { return ((nblocks_logical + 7) / 8) * 8; }

// Point outputs (slice, DeformSlice) are written once and not read back by
// the kernel: non-temporal stores keep them out of the L2.
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Store of 4 floats of a point row.  Non-temporal when a lane's part of the
// row is 16 bytes (fp32 inputs: a wave's store covers whole lines); with
// wider parts (bf16 inputs, 32 bytes a lane) one store instruction leaves
// gaps in every line, which the L2 has to merge, so those stay ordinary.
template <bool NT>
__device__ inline void store_row4(float* o, float a, float b, float c, float d) {
  if constexpr (NT)
    __builtin_nontemporal_store(f32x4_t{a, b, c, d}, reinterpret_cast<f32x4_t*>(o));
  else
    *reinterpret_cast<float4*>(o) = make_float4(a, b, c, d);
}

// f(std::integral_constant<int, i>) for i = 0 .. N-1, unrolled.
template <class F, int... I>
__device__ inline void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ inline void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Value of lane J of this lane's group of G lanes: a DPP row broadcast for
// G = 16 (a group is a row), a swizzle for G = 8 (bit mask mode: keep the
// group bits of the lane, set the low three to J).
template <int G, int J>
__device__ inline int32_t group_bcast(int32_t x) {
  static_assert(G == 16 || G == 8, "16- or 8-lane groups");
  if constexpr (G == 16) return __builtin_amdgcn_update_dpp(0, x, 0x150 + J, 0xF, 0xF, false);
  else return __builtin_amdgcn_ds_swizzle(x, 0x18 | (J << 5));
}

// Value of lane ^ OFF: DPP for partners inside a 16-lane row that DPP can
// name (xor 1 and 2 by quad permutation, xor 8 as a rotation by 8), a
// swizzle for xor 4 and 16 (within 32 lanes), a permute across halves.
template <int OFF>
__device__ inline float xor_lane(float v) {
  const int x = __float_as_int(v);
  if constexpr (OFF == 1) return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));
  else if constexpr (OFF == 2) return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));
  else if constexpr (OFF == 8) return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false));
  else if constexpr (OFF == 4 || OFF == 16) return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (OFF << 10)));
  else return __shfl_xor(v, OFF);
}

// Sum over the LPR lanes of a group, every lane receiving it.
template <int LPR>
__device__ inline float group_sum(float v) {
  if constexpr (LPR > 1) v += xor_lane<1>(v);
  if constexpr (LPR > 2) v += xor_lane<2>(v);
  if constexpr (LPR > 4) v += xor_lane<4>(v);
  if constexpr (LPR > 8) v += xor_lane<8>(v);
  if constexpr (LPR > 16) v += xor_lane<16>(v);
  if constexpr (LPR > 32) v += xor_lane<32>(v);
  return v;
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
      w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(base) + elem) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Splat (Eq. splat) as a gather over the point lists J_v, which are stored
// back to back (entries grouped by vertex).  The entry array is cut into
// chunks of `chunk` entries and each chunk goes to one lane group, so the
// work is balanced however skewed the vertex degrees are (a LiDAR vertex next
// to the sensor can hold thousands of points).  A vertex whose list lies
// inside one chunk is finished there.  A vertex cut by chunk boundaries
// leaves pieces: a head piece in a chunk it continues into, a tail piece in
// the chunk where it starts.  The G = kBlock/LPR consecutive chunks of a
// workgroup (its span) put their pieces in LDS and the workgroup joins them
// in chunk order: a vertex that starts and ends in the span is finished
// there; the piece of the vertex the span starts inside and the piece of the
// vertex that runs past its end go to global memory as the span's head and
// tail partials, which k_splat_finish adds in span order.  No float
// atomics; the summation order is fixed.
template <bool BF16, int LPR, int Q>
__device__ inline void splat_store(int32_t v, const float (&acc)[Q][Chunk<BF16>::N], float ws, int lane,
                                   int nchunk, int normalize, void* vals, int64_t ld_vals, float* wsum) {
  using Ch = Chunk<BF16>;
  const float scale = normalize ? (ws > 0.f ? 1.0f / ws : 0.f) : 1.0f;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int ch = lane + q * LPR;
    if (ch < nchunk) {
      Ch o;
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) o.v[i] = acc[q][i] * scale;
      o.store(vals, static_cast<int64_t>(v) * ld_vals + static_cast<int64_t>(ch) * Ch::N);
    }
  }
  if (wsum && lane == 0) wsum[v] = ws;
}

// row c of a C-wide partial array (global or LDS) and its weight
template <bool BF16, int LPR, int Q>
__device__ inline void splat_partial(float* part, float* part_w, int64_t c, int slot,
                                     const float (&acc)[Q][Chunk<BF16>::N], float ws, int lane, int C) {
  using Ch = Chunk<BF16>;
  const int nchunk = C / Ch::N;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int ch = lane + q * LPR;
    if (ch < nchunk) {
      float* dst = part + c * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
      for (int i = 0; i < Ch::N; i += 4)
        *reinterpret_cast<float4*>(dst + i) = make_float4(acc[q][i], acc[q][i + 1], acc[q][i + 2], acc[q][i + 3]);
    }
  }
  if (lane == 0) part_w[2 * c + slot] = ws;
}

template <bool BF16, int LPR, int Q>
__device__ inline void splat_add(float (&acc)[Q][Chunk<BF16>::N], const float* part, int64_t c, int lane, int C) {
  using Ch = Chunk<BF16>;
  const int nchunk = C / Ch::N;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int ch = lane + q * LPR;
    if (ch < nchunk) {
      const float* src = part + c * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
      for (int i = 0; i < Ch::N; i += 4) {
        const float4 x = *reinterpret_cast<const float4*>(src + i);
        acc[q][i] += x.x;
        acc[q][i + 1] += x.y;
        acc[q][i + 2] += x.z;
        acc[q][i + 3] += x.w;
      }
    }
  }
}

// What a list entry e = 4p + k adds to its vertex's row.  The splat adds
// w_e f_p (and w_e to the weight sum).
template <bool BF16, int LPR, int Q, int B>
struct WeightedRows {
  using Ch = Chunk<BF16>;
  const float* entry_w;
  const void* feat;
  int64_t ld_feat;
  struct Batch {
    float wt[B];
    Ch f[B][Q];
  };
  static constexpr bool kGivenWeights = true;   // the kernel may load entry_w itself
  __device__ inline void init(int, int) {}
  __device__ inline void load_given(Batch& bt, int j, float w, int32_t e, bool in, int lane, int nchunk) const {
    bt.wt[j] = in ? w : 0.f;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int ch = lane + q * LPR;
      if (in && ch < nchunk)
        bt.f[j][q].load(feat, static_cast<int64_t>(e >> 2) * ld_feat + static_cast<int64_t>(ch) * Ch::N);
      else
#pragma unroll
        for (int i = 0; i < Ch::N; ++i) bt.f[j][q].v[i] = 0.f;
    }
  }
  __device__ inline void load(Batch& bt, int j, int64_t s, int32_t e, bool in, int lane, int nchunk) const {
    bt.wt[j] = in ? entry_w[s] : 0.f;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int ch = lane + q * LPR;
      if (in && ch < nchunk)
        bt.f[j][q].load(feat, static_cast<int64_t>(e >> 2) * ld_feat + static_cast<int64_t>(ch) * Ch::N);
      else
#pragma unroll
        for (int i = 0; i < Ch::N; ++i) bt.f[j][q].v[i] = 0.f;
    }
  }
  __device__ inline float add(const Batch& bt, int j, float (&acc)[Q][Ch::N]) const {
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[q][i] += bt.wt[j] * bt.f[j][q].v[i];
    return bt.wt[j];
  }
};

// DeformSlice backward, what entry e = (p, k) adds to dL/dx of its vertex:
//   alpha_e g_p + wv * (beta_e - [argmax_c(p) = k] gamma_e)
// with coef[e] = (alpha_e, beta_e, gamma_e, 0) and am[p][c] the vertex slot
// holding channel c's maximum (fp32 only).
template <int LPR, int Q, int B>
struct DeformGradRows {
  using Ch = Chunk<false>;
  static constexpr bool kGivenWeights = false;
  const float* g;
  int64_t ld_g;
  const float4* coef;
  const uint8_t* am;
  const float* wv;
  int C;
  float wvc[Q][4];
  struct Batch {
    float4 cf[B];
    int k[B];
    Ch f[B][Q];
    uint32_t m[B][Q];
  };
  __device__ inline void init(int lane, int nchunk) {
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int ch = lane + q * LPR;
#pragma unroll
      for (int i = 0; i < 4; ++i) wvc[q][i] = ch < nchunk ? wv[4 * ch + i] : 0.f;
    }
  }
  __device__ inline void load(Batch& bt, int j, int64_t, int32_t e, bool in, int lane, int nchunk) const {
    bt.cf[j] = in ? coef[e] : make_float4(0.f, 0.f, 0.f, 0.f);
    bt.k[j] = e & 3;
    const int64_t p = e >> 2;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int ch = lane + q * LPR;
      if (in && ch < nchunk) {
        bt.f[j][q].load(g, p * ld_g + 4 * ch);
        bt.m[j][q] = *reinterpret_cast<const uint32_t*>(am + p * C + 4 * ch);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) bt.f[j][q].v[i] = 0.f;
        bt.m[j][q] = 0xffffffffu;
      }
    }
  }
  __device__ inline float add(const Batch& bt, int j, float (&acc)[Q][4]) const {
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool mx = ((bt.m[j][q] >> (8 * i)) & 0xffu) == static_cast<uint32_t>(bt.k[j]);
        acc[q][i] += bt.cf[j].x * bt.f[j][q].v[i] + wvc[q][i] * (bt.cf[j].y - (mx ? bt.cf[j].z : 0.f));
      }
    return 0.f;
  }
};

// LDS of k_splat_chunks: head and tail pieces of the G chunks, their weights
// and flags.
inline size_t splat_lds_bytes(int lpr, int C) {
  const int G = 256 / lpr;
  return sizeof(float) * (2 * static_cast<size_t>(G) * C + 2 * G) + sizeof(int32_t) * G;
}

template <bool BF16, int LPR, int Q, int B, class Rows>
__global__ void __launch_bounds__(kBlock)
k_splat_chunks(const int32_t* __restrict__ offsets, const int32_t* __restrict__ entries, Rows rows,
               const int32_t* __restrict__ chunk_first, int chunk, int64_t n, int64_t total, int C, int normalize,
               void* __restrict__ vals, int64_t ld_vals, float* __restrict__ wsum,
               float* __restrict__ part_head, float* __restrict__ part_tail, float* __restrict__ part_w,
               unsigned nblk) {
  using Ch = Chunk<BF16>;
  constexpr int G = kBlock / LPR;
  extern __shared__ __align__(16) float sm[];
  float* sh_head = sm;                 // [G][C]
  float* sh_tail = sm + G * C;         // [G][C]
  float* sh_w = sm + 2 * G * C;        // [G][2]
  int32_t* sh_flag = reinterpret_cast<int32_t*>(sh_w + 2 * G);  // bit 0 head piece, bit 1 tail piece
  const int lane = threadIdx.x & (LPR - 1);
  const int g = threadIdx.x / LPR;
  // XCD-contiguous span order (see xcd_item)
  const unsigned b = blockIdx.x;
  const int64_t span = static_cast<int64_t>(b % 8) * ((nblk + 7) / 8) + b / 8;
  const int64_t c0 = span * G;
  if (c0 * chunk >= total) return;     // whole workgroup
  const int64_t c = c0 + g;
  const int64_t s0 = c * chunk;
  const int64_t s1 = min(s0 + static_cast<int64_t>(chunk), total);
  const int64_t span_end = min((c0 + G) * static_cast<int64_t>(chunk), total);
  const int nchunk = C / Ch::N;
  rows.init(lane, nchunk);
  if (lane == 0) sh_flag[g] = 0;
  int32_t tail_v = -1, tail_ve = 0;    // vertex of this chunk's tail piece
  int32_t head_ve = 0;                 // end of the vertex the chunk starts inside
  if (s0 < total) {
    int32_t v = chunk_first[c];
    // window of list ends for the next LPR vertices
    int32_t v_win = v;
    int32_t win = offsets[min(static_cast<int64_t>(v) + 1 + lane, n)];
    int32_t vb = offsets[v];
    int32_t ve = __shfl(win, 0, LPR);
    head_ve = ve;
    float acc[Q][Ch::N];
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[q][i] = 0.f;
    float ws = 0.f;
    // what entry s (and the batch slot j it sits in) adds: the vertex's
    // running sum, and at the vertex's last entry (or the chunk's) its row or
    // piece
    auto consume = [&](const typename Rows::Batch& bt, int j, int64_t s) {
      ws += rows.add(bt, j, acc);
      const int64_t nxt = s + 1;
      if (nxt == ve || nxt == s1) {
        if (vb >= s0 && ve <= s1) {
          splat_store<BF16, LPR, Q>(v, acc, ws, lane, nchunk, normalize, vals, ld_vals, wsum);
        } else if (vb < s0) {
          splat_partial<BF16, LPR, Q>(sh_head, sh_w, g, 0, acc, ws, lane, C);
          if (lane == 0) sh_flag[g] |= 1;
        } else {
          splat_partial<BF16, LPR, Q>(sh_tail, sh_w, g, 1, acc, ws, lane, C);
          if (lane == 0) sh_flag[g] |= 2;
          tail_v = v;
          tail_ve = ve;
        }
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
          for (int i = 0; i < Ch::N; ++i) acc[q][i] = 0.f;
        ws = 0.f;
        if (nxt == ve && nxt < s1) {
          v += 1;
          vb = ve;
          if (v - v_win >= LPR) {
            v_win = v;
            win = offsets[min(static_cast<int64_t>(v) + 1 + lane, n)];
          }
          ve = __shfl(win, v - v_win, LPR);
        }
      }
    };
    if constexpr ((LPR == 16 || LPR == 8) && Rows::kGivenWeights) {
      // LPR entries at a time: lane i loads the index and weight of entry i,
      // and a broadcast inside the lane group (DPP or swizzle) hands entry
      // j's to the whole group; the next LPR are loaded while this round's
      // rows arrive
      int32_t E = s0 + lane < s1 ? entries[s0 + lane] : 0;
      float Wt = s0 + lane < s1 ? rows.entry_w[s0 + lane] : 0.f;
      for (int64_t sb = s0; sb < s1; sb += LPR) {
        const int64_t nx = sb + LPR + lane;
        const int32_t En = nx < s1 ? entries[nx] : 0;
        const float Wn = nx < s1 ? rows.entry_w[nx] : 0.f;
        static_for<LPR / B>([&](auto h_c) {
          constexpr int J0 = decltype(h_c)::value * B;
          if (sb + J0 < s1) {
            typename Rows::Batch bt;
            static_for<B>([&](auto j_c) {
              constexpr int J = decltype(j_c)::value;
              const int32_t e = group_bcast<LPR, J0 + J>(E);
              const float w = __int_as_float(group_bcast<LPR, J0 + J>(__float_as_int(Wt)));
              rows.load_given(bt, J, w, e, sb + J0 + J < s1, lane, nchunk);
            });
#pragma unroll
            for (int j = 0; j < B; ++j) {
              if (sb + J0 + j >= s1) break;
              consume(bt, j, sb + J0 + j);
            }
          }
        });
        E = En;
        Wt = Wn;
      }
    } else {
      // the entries of the next batch are loaded while this batch's rows
      // arrive and are added
      int32_t e[B];
#pragma unroll
      for (int j = 0; j < B; ++j) e[j] = s0 + j < s1 ? entries[s0 + j] : 0;
      for (int64_t s = s0; s < s1; s += B) {
        typename Rows::Batch bt;
#pragma unroll
        for (int j = 0; j < B; ++j) rows.load(bt, j, s + j, e[j], s + j < s1, lane, nchunk);
#pragma unroll
        for (int j = 0; j < B; ++j) e[j] = s + B + j < s1 ? entries[s + B + j] : 0;
#pragma unroll
        for (int j = 0; j < B; ++j) {
          if (s + j >= s1) break;
          consume(bt, j, s + j);
        }
      }
    }
  }
  __syncthreads();
  // join the pieces of the span in chunk order
  float acc[Q][Ch::N];
  if (tail_v >= 0) {
    // vertex starting in chunk g: its tail piece, then the head pieces of the
    // following chunks it runs into
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[q][i] = 0.f;
    splat_add<BF16, LPR, Q>(acc, sh_tail, g, lane, C);
    float ws = sh_w[2 * g + 1];
    for (int g2 = g + 1; g2 < G && (c0 + g2) * chunk < tail_ve; ++g2) {
      splat_add<BF16, LPR, Q>(acc, sh_head, g2, lane, C);
      ws += sh_w[2 * g2];
    }
    if (tail_ve <= span_end)
      splat_store<BF16, LPR, Q>(tail_v, acc, ws, lane, nchunk, normalize, vals, ld_vals, wsum);
    else
      splat_partial<BF16, LPR, Q>(part_tail, part_w, span, 1, acc, ws, lane, C);
  }
  if (g == 0 && (sh_flag[0] & 1)) {
    // the vertex the span starts inside: head pieces of the chunks it covers
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[q][i] = 0.f;
    float ws = 0.f;
    for (int g2 = 0; g2 < G && (c0 + g2) * chunk < head_ve; ++g2) {
      splat_add<BF16, LPR, Q>(acc, sh_head, g2, lane, C);
      ws += sh_w[2 * g2];
    }
    splat_partial<BF16, LPR, Q>(part_head, part_w, span, 0, acc, ws, lane, C);
  }
}

// Vertices cut by span boundaries: the span in which a vertex's list starts
// adds its tail partial and the head partials of the following spans.
template <bool BF16, int LPR, int Q>
__global__ void __launch_bounds__(kBlock)
k_splat_finish(const int32_t* __restrict__ offsets, const int32_t* __restrict__ chunk_first, int64_t span_len,
               int chunks_per_span, int64_t nspans, int C, int normalize, void* __restrict__ vals, int64_t ld_vals,
               float* __restrict__ wsum, const float* __restrict__ part_head, const float* __restrict__ part_tail,
               const float* __restrict__ part_w) {
  using Ch = Chunk<BF16>;
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / LPR;
  if (c + 1 >= nspans) return;
  const int64_t s0 = c * span_len, s1 = s0 + span_len;
  const int32_t v = chunk_first[(c + 1) * chunks_per_span];
  const int32_t vb = offsets[v];
  if (!(vb < s1 && vb >= s0)) return;
  const int32_t ve = offsets[v + 1];
  const int64_t last = (static_cast<int64_t>(ve) - 1) / span_len;
  const int nchunk = C / Ch::N;
  float acc[Q][Ch::N];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int i = 0; i < Ch::N; ++i) acc[q][i] = 0.f;
  splat_add<BF16, LPR, Q>(acc, part_tail, c, lane, C);
  float ws = part_w[2 * c + 1];
#pragma unroll 8
  for (int64_t c2 = c + 1; c2 <= last; ++c2) {
    splat_add<BF16, LPR, Q>(acc, part_head, c2, lane, C);
    ws += part_w[2 * c2];
  }
  splat_store<BF16, LPR, Q>(v, acc, ws, lane, nchunk, normalize, vals, ld_vals, wsum);
}

// Slice (Eq. slice): out_p = sum_k b_pk x_{idx_pk}.  A lane group takes two
// consecutive points and issues the loads of both before using them (twice
// the bytes in flight per lane).  A vertex slot without a vertex (a lattice
// the build flagged) reads row 0 with weight 0, so that the loads are issued
// without branches.
template <bool BF16, int LPR>
__global__ void __launch_bounds__(kBlock)
k_slice(const int4* __restrict__ idx, const float4* __restrict__ w, int64_t m,
        const void* __restrict__ vals, int64_t ld_vals, int C, float* __restrict__ out, unsigned nblk) {
  using Ch = Chunk<BF16>;
  constexpr int PP = 2;
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t p0 = PP * xcd_item<LPR>(nblk);
  if (p0 >= m) return;
  int32_t vi[PP][4];
  float bw[PP][4];
#pragma unroll
  for (int u = 0; u < PP; ++u) {
    const int64_t p = min(p0 + u, m - 1);
    const int4 iv = idx[p];
    const float4 wv = w[p];
    vi[u][0] = max(iv.x, 0); vi[u][1] = max(iv.y, 0); vi[u][2] = max(iv.z, 0); vi[u][3] = max(iv.w, 0);
    bw[u][0] = iv.x < 0 ? 0.f : wv.x;
    bw[u][1] = iv.y < 0 ? 0.f : wv.y;
    bw[u][2] = iv.z < 0 ? 0.f : wv.z;
    bw[u][3] = iv.w < 0 ? 0.f : wv.w;
  }
  const int nchunk = C / Ch::N;
  for (int ch = lane; ch < nchunk; ch += LPR) {
    Ch x[PP][4];
#pragma unroll
    for (int u = 0; u < PP; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        x[u][k].load(vals, static_cast<int64_t>(vi[u][k]) * ld_vals + static_cast<int64_t>(ch) * Ch::N);
#pragma unroll
    for (int u = 0; u < PP; ++u) {
      if (p0 + u >= m) break;
      float acc[Ch::N];
#pragma unroll
      for (int i = 0; i < Ch::N; ++i) acc[i] = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < Ch::N; ++i) acc[i] += bw[u][k] * x[u][k].v[i];
      float* o = out + (p0 + u) * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
      for (int i = 0; i < Ch::N; i += 4)
        store_row4<Ch::N == 4>(o + i, acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
    }
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
               float beta, float* __restrict__ out, float4* __restrict__ delta, float* __restrict__ plain,
               unsigned nblk) {
  using Ch = Chunk<BF16>;
  const int lane = threadIdx.x & (LPR - 1);
  const int64_t p = xcd_item<LPR>(nblk);
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
  for (int k = 0; k < 4; ++k) part[k] = group_sum<LPR>(part[k]);
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
      store_row4<Ch::N == 4>(o + i, r[0], r[1], r[2], r[3]);
    }
    if (plain) {
      // the plain slice of the same rows (Eq. slice), in the order of k_slice
      float* o2 = plain + p * C + static_cast<int64_t>(ch) * Ch::N;
#pragma unroll
      for (int i = 0; i < Ch::N; i += 4) {
        float r[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float a = 0.f;
#pragma unroll
          for (int k = 0; k < 4; ++k) a += bw[k] * x[q][k][i + u];
          r[u] = a;
        }
        store_row4<Ch::N == 4>(o2 + i, r[0], r[1], r[2], r[3]);
      }
    }
  }
}

// lanes per row: enough 16-byte chunks to cover C, at most 64 (a wavefront)
// One exchange of the reduce-scatter in k_deform_classify: lanes whose bit
// OFF is set keep the upper LEN values, the others the lower LEN, and each
// adds the half its partner gives away.
// One exchange of the reduce-scatter in k_deform_classify: lanes whose bit
// OFF is set keep the upper LEN values, the others the lower LEN, and each
// adds the half its partner gives away.

// One exchange of the reduce-scatter in k_deform_classify: lanes whose bit
// OFF is set keep the upper LEN values, the others the lower LEN, and each
// adds the half its partner gives away; blk gathers the kept halves' bits.
template <int OFF, int LEN, int KP>
__device__ inline void reduce_scatter_step(float (&lg)[KP], int lane, int& blk) {
  const bool up = (lane & OFF) != 0;
#pragma unroll
  for (int i = 0; i < LEN; ++i) {
    const float give = up ? lg[i] : lg[i + LEN];
    const float keep = up ? lg[i + LEN] : lg[i];
    lg[i] = keep + xor_lane<OFF>(give);
  }
  blk = 2 * blk + (up ? 1 : 0);
}


// DeformSlice fused with the last linear classification layer
// (Implementation): the DeformSlice row of a point is formed in registers as
// in k_deform_slice and multiplied by Wc (K x C, staged in LDS); the KP >= K
// logit partials of a lane group are summed by a reduce-scatter, after which
// each lane holds KP / LPR finished classes (the block its exchange bits
// name).  The high-dimensional per-point row is never stored.
template <bool BF16, int LPR, int CPL, int KP>
__global__ void __launch_bounds__(kBlock)
k_deform_classify(const int4* __restrict__ idx, const float4* __restrict__ w, int64_t m,
                  const void* __restrict__ vals, int64_t ld_vals, int C, const float* __restrict__ wvec, float beta,
                  const float* __restrict__ Wc, const float* __restrict__ bc, int K, float* __restrict__ out,
                  unsigned nblk) {
  using Ch = Chunk<BF16>;
  extern __shared__ __align__(16) float wl[];   // [K][C]
  for (int i = threadIdx.x; i < K * C; i += kBlock) wl[i] = Wc[i];
  __syncthreads();
  const int lane = threadIdx.x & (LPR - 1);
  const int nchunk = C / Ch::N;
  // The weights are staged once per workgroup, which then walks a
  // contiguous range of the nblk logical blocks (each XCD a contiguous
  // share of the ranges, as xcd_item).
  const unsigned G = gridDim.x;   // a multiple of 8
  const unsigned r = (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8;
  const unsigned per = (nblk + G - 1) / G;
  const unsigned lb1 = min((r + 1) * per, nblk);
  for (unsigned lb = r * per; lb < lb1; ++lb) {
  const int64_t p = (static_cast<int64_t>(lb) * kBlock + threadIdx.x) / LPR;
  const bool live = p < m;
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
  for (int k = 0; k < 4; ++k) part[k] = group_sum<LPR>(part[k]);
  float coef[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) coef[k] = bw[k] + tanhf(beta + part[k]);
  float lg[KP];
#pragma unroll
  for (int j = 0; j < KP; ++j) lg[j] = 0.f;
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int ch = lane + q * LPR;
    if (!(live && ch < nchunk)) continue;
#pragma unroll
    for (int i = 0; i < Ch::N; i += 4) {
      float f[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        f[u] = coef[0] * x[q][0][i + u] + coef[1] * x[q][1][i + u] + coef[2] * x[q][2][i + u] +
               coef[3] * x[q][3][i + u];
#pragma unroll
      for (int j = 0; j < KP; ++j) {
        if (j >= K) break;
        const float4 wv4 = *reinterpret_cast<const float4*>(wl + j * C + ch * Ch::N + i);
        lg[j] += wv4.x * f[0] + wv4.y * f[1] + wv4.z * f[2] + wv4.w * f[3];
      }
    }
  }
  // the exchanges in the order of their cost (cheap ones move the most
  // values); blk = the class block this lane keeps
  int blk = 0;
  constexpr int S = (LPR >= 2) + (LPR >= 4) + (LPR >= 8) + (LPR >= 16) + (LPR >= 32) + (LPR >= 64);
  static_assert((KP >> S) >= 1, "at least one class per lane");
  if constexpr (LPR >= 2) reduce_scatter_step<1, (KP >> 1)>(lg, lane, blk);
  if constexpr (LPR >= 4) reduce_scatter_step<2, (KP >> 2)>(lg, lane, blk);
  if constexpr (LPR >= 16) reduce_scatter_step<8, (KP >> 3)>(lg, lane, blk);
  if constexpr (LPR >= 8) reduce_scatter_step<4, (KP >> (LPR >= 16 ? 4 : 3))>(lg, lane, blk);
  if constexpr (LPR >= 32) reduce_scatter_step<16, (KP >> 5)>(lg, lane, blk);
  if constexpr (LPR >= 64) reduce_scatter_step<32, (KP >> 6)>(lg, lane, blk);
  if (live) {
    constexpr int OWN = KP / LPR;
#pragma unroll
    for (int i = 0; i < OWN; ++i) {
      const int j = blk * OWN + i;
      if (j < K) out[p * K + j] = lg[i] + (bc ? bc[j] : 0.f);
    }
  }
  }
}

// DeformSlice backward, per point (C channels over LPR lanes, CPL 16-byte
// chunks per lane, as in the forward), with g = dL/dout_p:
//   q_k = b_k x_k; am_c = the first slot k whose float32 q_k is maximal,
//   M_c = q_{am_c}; s_k = beta + (q_k - M) . wv; db_k = tanh(s_k);
//   a_k = g . x_k; e_k = a_k (1 - db_k^2) (= dL/ds_k).
// It writes coef[4p + k] = (b_k + db_k, e_k b_k, (sum_j e_j) b_k, 0) and
// am[p][c] for the gather over J_v, and adds sum_k e_k (q_k - M) (dL/dwv) and
// sum_k e_k (dL/dbeta) into per-workgroup partials: the workgroups stride
// over the points, sum in registers, then over their lane groups in a fixed
// order.
template <int LPR, int CPL>
__global__ void __launch_bounds__(kBlock)
k_deform_bwd_point(const int4* __restrict__ idx, const float4* __restrict__ w, int64_t m,
                   const float* __restrict__ vals, int64_t ld_vals, int C, const float* __restrict__ wvec, float beta,
                   const float* __restrict__ dout, int64_t ld_dout, float4* __restrict__ coef,
                   uint8_t* __restrict__ am, float* __restrict__ part_wv, float* __restrict__ part_beta) {
  constexpr int G = kBlock / LPR;
  __shared__ float red[kBlock * CPL * 4];   // [group][channel], G * C <= this
  __shared__ float red_b[G];
  const int lane = threadIdx.x & (LPR - 1), grp = threadIdx.x / LPR;
  const int nchunk = C / 4;
  float wacc[CPL][4];
#pragma unroll
  for (int q = 0; q < CPL; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) wacc[q][i] = 0.f;
  float bacc = 0.f;
  const int64_t groups = (m + G - 1) / G;
  for (int64_t it = blockIdx.x; it < groups; it += gridDim.x) {
    const int64_t p = it * G + grp;
    const bool live = p < m;
    int4 iv = make_int4(0, 0, 0, 0);
    float4 wq = make_float4(0.f, 0.f, 0.f, 0.f);
    if (live) { iv = idx[p]; wq = w[p]; }
    const int32_t vi[4] = {iv.x, iv.y, iv.z, iv.w};
    const float bw[4] = {wq.x, wq.y, wq.z, wq.w};
    float x[CPL][4][4], gv[CPL][4], mx[CPL][4];
    float sp[4] = {0.f, 0.f, 0.f, 0.f}, ap[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      const int ch = lane + q * LPR;
      const bool on = live && ch < nchunk;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (on) v = *reinterpret_cast<const float4*>(vals + static_cast<int64_t>(vi[k]) * ld_vals + 4 * ch);
        x[q][k][0] = v.x; x[q][k][1] = v.y; x[q][k][2] = v.z; x[q][k][3] = v.w;
      }
      float4 gg = make_float4(0.f, 0.f, 0.f, 0.f);
      if (on) gg = *reinterpret_cast<const float4*>(dout + p * ld_dout + 4 * ch);
      gv[q][0] = gg.x; gv[q][1] = gg.y; gv[q][2] = gg.z; gv[q][3] = gg.w;
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float wc = on ? wvec[4 * ch + i] : 0.f;
        float qk[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) qk[k] = bw[k] * x[q][k][i];
        float best = qk[0];
        uint32_t a = 0;
#pragma unroll
        for (int k = 1; k < 4; ++k)
          if (qk[k] > best) {
            best = qk[k];
            a = static_cast<uint32_t>(k);
          }
        mx[q][i] = best;
        word |= a << (8 * i);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          sp[k] += (qk[k] - best) * wc;
          ap[k] += gv[q][i] * x[q][k][i];
        }
      }
      if (on) *reinterpret_cast<uint32_t*>(am + p * C + 4 * ch) = word;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      sp[k] = group_sum<LPR>(sp[k]);
      ap[k] = group_sum<LPR>(ap[k]);
    }
    float e[4], esum = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float db = tanhf(beta + sp[k]);
      e[k] = ap[k] * (1.f - db * db);
      esum += e[k];
      sp[k] = db;
    }
    if (!live) continue;
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) coef[4 * p + k] = make_float4(bw[k] + sp[k], e[k] * bw[k], esum * bw[k], 0.f);
      bacc += esum;
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k) a += e[k] * (bw[k] * x[q][k][i] - mx[q][i]);
        wacc[q][i] += a;
      }
  }
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int ch = lane + q * LPR;
    if (ch < nchunk)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[grp * C + 4 * ch + i] = wacc[q][i];
  }
  if (lane == 0) red_b[grp] = bacc;
  __syncthreads();
  for (int c = threadIdx.x; c < C; c += kBlock) {
    float a = 0.f;
    for (int g2 = 0; g2 < G; ++g2) a += red[g2 * C + c];
    part_wv[static_cast<int64_t>(blockIdx.x) * C + c] = a;
  }
  if (threadIdx.x == 0) {
    float a = 0.f;
    for (int g2 = 0; g2 < G; ++g2) a += red_b[g2];
    part_beta[blockIdx.x] = a;
  }
}

// dL/dwv[c] (workgroup c < C) and dL/dbeta (workgroup C): the per-workgroup
// partials added by a fixed tree.
__global__ void __launch_bounds__(kBlock)
k_deform_bwd_reduce(const float* __restrict__ part_wv, const float* __restrict__ part_beta, int64_t nparts, int C,
                    float* __restrict__ dwv, float* __restrict__ dbeta) {
  __shared__ float sh[kBlock];
  const int c = blockIdx.x;
  float a = 0.f;
  for (int64_t b = threadIdx.x; b < nparts; b += kBlock) a += c < C ? part_wv[b * C + c] : part_beta[b];
  sh[threadIdx.x] = a;
  __syncthreads();
  for (int off = kBlock / 2; off > 0; off >>= 1) {
    if (static_cast<int>(threadIdx.x) < off) sh[threadIdx.x] += sh[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (c < C) dwv[c] = sh[0];
    else *dbeta = sh[0];
  }
}

inline int lanes_per_row(int C, bool bf16) {
  const int chunks = C / (bf16 ? 8 : 4);
  int l = 1;
  while (l < chunks && l < 64) l <<= 1;
  return l;
}

// Lane group of one row (one vertex list entry or one point) for the splat,
// DeformSlice, the fused classifier and the DeformSlice gradient's point
// pass: 64 fp32 channels take 8 lanes of two 16-byte chunks each (half the
// per-entry bookkeeping per channel), every other width one chunk per lane.
// DeformSlice and its gradient must agree: the gradient recomputes the
// offsets, and the same lane groups sum the dot products in the same order.
inline int point_lanes_per_row(int C, bool bf16) {
  return !bf16 && C / 4 == 16 ? 8 : lanes_per_row(C, bf16);
}

inline unsigned grid_for(int64_t rows, int lpr) {
  return static_cast<unsigned>((rows * lpr + kBlock - 1) / kBlock);
}

template <bool BF16, int LPR, int Q>
void splat_launch(const int32_t* off, const int32_t* ent, const float* ew, const int32_t* cf, int chunk, int64_t n, int64_t total,
                  const void* feat, int64_t ldf, int C, int norm, void* vals, int64_t ldv, float* wsum,
                  float* ph, float* pt, float* pw, hipStream_t s) {
  constexpr int B = 8 / Q;   // entries in flight per lane group (more would cost occupancy)
  constexpr int G = kBlock / LPR;
  const int64_t span_len = static_cast<int64_t>(G) * chunk;
  const int64_t nspans = (total + span_len - 1) / span_len;
  const unsigned nblk = static_cast<unsigned>(nspans);
  const size_t lds = splat_lds_bytes(LPR, C);
  using Rows = WeightedRows<BF16, LPR, Q, B>;
  static bool lds_limit_set = false;
  if (!lds_limit_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_splat_chunks<BF16, LPR, Q, B, Rows>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(splat_lds_bytes(LPR, LPR * Q * Chunk<BF16>::N)));
    lds_limit_set = true;
  }
  const Rows rows{ew, feat, ldf};
  launch((k_splat_chunks<BF16, LPR, Q, B, Rows>), dim3(xcd_grid(nblk)), dim3(kBlock), lds, s, off, ent, rows, cf,
         chunk, n, total, C, norm, vals, ldv, wsum, ph, pt, pw, nblk);
  if (nspans > 1)
    launch((k_splat_finish<BF16, LPR, Q>), dim3(grid_for(nspans, LPR)), dim3(kBlock), 0, s, off, cf,
                       span_len, G, nspans, C, norm, vals, ldv, wsum, ph, pt, pw);
}

template <bool BF16>
void splat_dispatch(int lpr, int q, const int32_t* off, const int32_t* ent, const float* ew,
                    const int32_t* cf, int chunk, int64_t n, int64_t total, const void* feat, int64_t ldf, int C, int norm,
                    void* vals, int64_t ldv, float* wsum, float* ph, float* pt, float* pw, hipStream_t s) {
#define SPLAT_CASE(L, QQ) \
  if (lpr == L && q == QQ) return splat_launch<BF16, L, QQ>(off, ent, ew, cf, chunk, n, total, feat, ldf, C, norm, vals, ldv, wsum, ph, pt, pw, s);
  SPLAT_CASE(1, 1) SPLAT_CASE(2, 1) SPLAT_CASE(4, 1) SPLAT_CASE(8, 1) SPLAT_CASE(16, 1)
  SPLAT_CASE(32, 1) SPLAT_CASE(64, 1) SPLAT_CASE(64, 2) SPLAT_CASE(64, 4) SPLAT_CASE(8, 2)
#undef SPLAT_CASE
}

template <int LPR, int Q>
void deform_grad_gather(const int32_t* off, const int32_t* ent, const int32_t* cf, int chunk, int64_t n,
                        int64_t total, const float* g, int64_t ldg, const float4* coef, const uint8_t* am,
                        const float* wv, int C, float* dx, int64_t ldx, float* ph, float* pt, float* pw,
                        hipStream_t s) {
  constexpr int B = 8 / Q;
  constexpr int G = kBlock / LPR;
  using Rows = DeformGradRows<LPR, Q, B>;
  const int64_t span_len = static_cast<int64_t>(G) * chunk;
  const int64_t nspans = (total + span_len - 1) / span_len;
  const unsigned nblk = static_cast<unsigned>(nspans);
  const size_t lds = splat_lds_bytes(LPR, C);
  static bool lds_limit_set = false;
  if (!lds_limit_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_splat_chunks<false, LPR, Q, B, Rows>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(splat_lds_bytes(LPR, LPR * Q * 4)));
    lds_limit_set = true;
  }
  Rows rows{g, ldg, coef, am, wv, C, {}};
  launch((k_splat_chunks<false, LPR, Q, B, Rows>), dim3(xcd_grid(nblk)), dim3(kBlock), lds, s, off, ent, rows, cf,
         chunk, n, total, C, 0, static_cast<void*>(dx), ldx, static_cast<float*>(nullptr), ph, pt, pw, nblk);
  if (nspans > 1)
    launch((k_splat_finish<false, LPR, Q>), dim3(grid_for(nspans, LPR)), dim3(kBlock), 0, s, off, cf, span_len, G,
           nspans, C, 0, static_cast<void*>(dx), ldx, static_cast<float*>(nullptr), static_cast<const float*>(ph),
           static_cast<const float*>(pt), static_cast<const float*>(pw));
}

void deform_grad_dispatch(int lpr, int q, const int32_t* off, const int32_t* ent, const int32_t* cf, int chunk,
                          int64_t n, int64_t total, const float* g, int64_t ldg, const float4* coef,
                          const uint8_t* am, const float* wv, int C, float* dx, int64_t ldx, float* ph, float* pt,
                          float* pw, hipStream_t s) {
#define DGRAD_CASE(L, QQ) \
  if (lpr == L && q == QQ) return deform_grad_gather<L, QQ>(off, ent, cf, chunk, n, total, g, ldg, coef, am, wv, C, dx, ldx, ph, pt, pw, s);
  DGRAD_CASE(1, 1) DGRAD_CASE(2, 1) DGRAD_CASE(4, 1) DGRAD_CASE(8, 1) DGRAD_CASE(16, 1)
  DGRAD_CASE(32, 1) DGRAD_CASE(64, 1) DGRAD_CASE(64, 2)
#undef DGRAD_CASE
}

template <int CPL>
void deform_bwd_point_dispatch(int lpr, unsigned grid, const int32_t* idx, const float* w, int64_t m,
                               const float* vals, int64_t ldv, int C, const float* wv, float beta, const float* dout,
                               int64_t ldo, float4* coef, uint8_t* am, float* pwv, float* pb, hipStream_t s) {
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
#define DPT_CASE(L) \
  if (lpr == L) return launch((k_deform_bwd_point<L, CPL>), dim3(grid), dim3(kBlock), 0, s, i4, w4, m, vals, ldv, C, wv, beta, dout, ldo, coef, am, pwv, pb);
  DPT_CASE(1) DPT_CASE(2) DPT_CASE(4) DPT_CASE(8) DPT_CASE(16) DPT_CASE(32) DPT_CASE(64)
#undef DPT_CASE
}

template <bool BF16>
void slice_dispatch(int lpr, const int32_t* idx, const float* w, int64_t m, const void* vals,
                    int64_t ldv, int C, float* out, hipStream_t s) {
  const unsigned nblk = grid_for((m + 1) / 2, lpr);   // two points per lane group
  const dim3 g(xcd_grid(nblk)), b(kBlock);
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  switch (lpr) {
    case 1: launch((k_slice<BF16, 1>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    case 2: launch((k_slice<BF16, 2>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    case 4: launch((k_slice<BF16, 4>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    case 8: launch((k_slice<BF16, 8>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    case 16: launch((k_slice<BF16, 16>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    case 32: launch((k_slice<BF16, 32>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
    default: launch((k_slice<BF16, 64>), g, b, 0, s, i4, w4, m, vals, ldv, C, out, nblk); break;
  }
}

template <bool BF16, int CPL>
void deform_dispatch(int lpr, const int32_t* idx, const float* w, int64_t m, const void* vals,
                     int64_t ldv, int C, const float* wv, float beta, float* out, float* delta, float* plain,
                     hipStream_t s) {
  const unsigned nblk = grid_for(m, lpr);
  const dim3 g(xcd_grid(nblk)), b(kBlock);
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  float4* d4 = reinterpret_cast<float4*>(delta);
  switch (lpr) {
    case 1: launch((k_deform_slice<BF16, 1, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    case 2: launch((k_deform_slice<BF16, 2, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    case 4: launch((k_deform_slice<BF16, 4, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    case 8: launch((k_deform_slice<BF16, 8, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    case 16: launch((k_deform_slice<BF16, 16, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    case 32: launch((k_deform_slice<BF16, 32, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
    default: launch((k_deform_slice<BF16, 64, CPL>), g, b, 0, s, i4, w4, m, vals, ldv, C, wv, beta, out, d4, plain, nblk); break;
  }
}

}  // namespace

// Largest channel count the gather kernels handle: 4 chunks per lane of a
// full wavefront for splat, 2 for DeformSlice; slice loops without limit.
int splat_max_channels(bool bf16) { return (bf16 ? 8 : 4) * 64 * 4; }
int deform_max_channels(bool bf16) { return (bf16 ? 8 : 4) * 64 * 2; }

// Partials of k_splat_chunks: a head and a tail row of C floats and two
// weights per span of kBlock/LPR chunks (sized for the smallest span, LPR =
// 64, whatever the channel count).
int64_t splat_partial_floats(int64_t total, int chunk, int C) {
  const int64_t span_len = static_cast<int64_t>(kBlock / 64) * chunk;
  const int64_t nspans = (total + span_len - 1) / span_len;
  return nspans * (2 * static_cast<int64_t>(C) + 2);
}

void launch_splat(const int32_t* offsets, const int32_t* entries, const float* entry_w,
                  const int32_t* chunk_first, int chunk, int64_t n, int64_t total, const void* feat, int64_t ld_feat, int C,
                  int bf16, int normalize, void* vals, int64_t ld_vals, float* wsum, float* partials,
                  hipStream_t s) {
  if (total <= 0) return;
  const int chunks = C / (bf16 ? 8 : 4);
  const int lpr = point_lanes_per_row(C, bf16 != 0);
  const int q = chunks <= lpr ? 1 : (chunks <= 2 * lpr ? 2 : 4);
  const int64_t span_len = static_cast<int64_t>(kBlock / lpr) * chunk;
  const int64_t nspans = (total + span_len - 1) / span_len;
  float* ph = partials;
  float* pt = partials + nspans * C;
  float* pw = partials + 2 * nspans * C;
  ScopedKernelTimer tm("splat", s);
  if (bf16) splat_dispatch<true>(lpr, q, offsets, entries, entry_w, chunk_first, chunk, n, total, feat, ld_feat, C, normalize, vals, ld_vals, wsum, ph, pt, pw, s);
  else splat_dispatch<false>(lpr, q, offsets, entries, entry_w, chunk_first, chunk, n, total, feat, ld_feat, C, normalize, vals, ld_vals, wsum, ph, pt, pw, s);
}

void launch_slice(const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ld_vals,
                  int C, int bf16, float* out, hipStream_t s) {
  if (m <= 0) return;
  const int lpr = lanes_per_row(C, bf16 != 0);
  ScopedKernelTimer tm("slice", s);
  if (bf16) slice_dispatch<true>(lpr, idx, w, m, vals, ld_vals, C, out, s);
  else slice_dispatch<false>(lpr, idx, w, m, vals, ld_vals, C, out, s);
}

template <bool BF16, int CPL, int KP>
void deform_classify_dispatch(int lpr, const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ldv,
                              int C, const float* wv, float beta, const float* Wc, const float* bc, int K,
                              float* out, hipStream_t s) {
  const unsigned nblk = grid_for(m, lpr);
  const dim3 g(std::min(xcd_grid(nblk), kClassifyGrid)), b(kBlock);
  const int4* i4 = reinterpret_cast<const int4*>(idx);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  const uint32_t lds = static_cast<uint32_t>(4 * K * C);
#define DCL_CASE(L)                                                                                              \
  if (lpr == L) {                                                                                                \
    static bool set = false;                                                                                     \
    if (!set) {                                                                                                  \
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_deform_classify<BF16, L, CPL, KP>),               \
                                hipFuncAttributeMaxDynamicSharedMemorySize, 4 * kClassifyMaxWeights);           \
      set = true;                                                                                                \
    }                                                                                                            \
    return launch((k_deform_classify<BF16, L, CPL, KP>), g, b, lds, s, i4, w4, m, vals, ldv, C, wv, beta, Wc, bc, K, \
                  out, nblk);                                                                                    \
  }
  if constexpr (KP >= 64) { DCL_CASE(64) }
  DCL_CASE(1) DCL_CASE(2) DCL_CASE(4) DCL_CASE(8) DCL_CASE(16) DCL_CASE(32)
#undef DCL_CASE
}

int deform_classify_max_classes() { return 64; }
int deform_classify_max_weights() { return kClassifyMaxWeights; }

void launch_deform_classify(const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ld_vals, int C,
                            int bf16, const float* wv, float beta, const float* Wc, const float* bc, int K, float* out,
                            hipStream_t s) {
  if (m <= 0) return;
  const int chunks = C / (bf16 ? 8 : 4);
  const int lpr = point_lanes_per_row(C, bf16 != 0);
  ScopedKernelTimer tm("deform_slice", s);
  const bool two = chunks > lpr;
  const bool kp64 = K > 32 || lpr > 32;
#define DCL_GO(BFV, CPLV)                                                                                          \
  (kp64 ? deform_classify_dispatch<BFV, CPLV, 64>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, Wc, bc, K, out, s)  \
        : deform_classify_dispatch<BFV, CPLV, 32>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, Wc, bc, K, out, s))
  if (bf16) {
    if (two) DCL_GO(true, 2);
    else DCL_GO(true, 1);
  } else {
    if (two) DCL_GO(false, 2);
    else DCL_GO(false, 1);
  }
#undef DCL_GO
}

// Work space of launch_deform_slice_backward, in bytes.
int64_t deform_backward_workspace_bytes(int64_t m, int C, int64_t total, int chunk) {
  return 16 * 4 * m + m * C + 4 * (kDeformBwdGrid * (static_cast<int64_t>(C) + 1)) +
         4 * splat_partial_floats(total, chunk, C) + 64;
}

void launch_deform_slice_backward(const int32_t* idx, const float* w, int64_t m, const int32_t* offsets,
                                  const int32_t* entries, const int32_t* chunk_first, int chunk, int64_t n,
                                  int64_t total, const float* vals, int64_t ld_vals, int C, const float* wv,
                                  float beta, const float* dout, int64_t ld_dout, float* dvals, int64_t ld_dvals,
                                  float* dwv, float* dbeta, void* work, hipStream_t s) {
  ScopedKernelTimer tm("deform_bwd", s);
  if (m <= 0 || n <= 0) {
    // no point: dL/dwv and dL/dbeta are empty sums
    launch(k_deform_bwd_reduce, dim3(static_cast<unsigned>(C + 1)), dim3(kBlock), 0, s,
           static_cast<const float*>(nullptr), static_cast<const float*>(nullptr), static_cast<int64_t>(0), C, dwv,
           dbeta);
    return;
  }
  char* wp = static_cast<char*>(work);
  float4* coef = reinterpret_cast<float4*>(wp);
  wp += 16 * 4 * m;
  float* pwv = reinterpret_cast<float*>(wp);
  wp += 4 * kDeformBwdGrid * static_cast<int64_t>(C);
  float* pb = reinterpret_cast<float*>(wp);
  wp += 4 * kDeformBwdGrid;
  float* parts = reinterpret_cast<float*>(wp);
  wp += 4 * splat_partial_floats(total, chunk, C);
  uint8_t* am = reinterpret_cast<uint8_t*>(wp);
  // the point pass on the forward's lane groups (the same offsets); the
  // gather over the vertex lists on one chunk per lane
  const int plpr = point_lanes_per_row(C, false);
  const int lpr = lanes_per_row(C, false);
  const int chunks = C / 4;
  const int G = kBlock / plpr;
  const int64_t groups = (m + G - 1) / G;
  const unsigned grid = static_cast<unsigned>(std::min<int64_t>(groups, kDeformBwdGrid));
  if (chunks > plpr)
    deform_bwd_point_dispatch<2>(plpr, grid, idx, w, m, vals, ld_vals, C, wv, beta, dout, ld_dout, coef, am, pwv, pb, s);
  else
    deform_bwd_point_dispatch<1>(plpr, grid, idx, w, m, vals, ld_vals, C, wv, beta, dout, ld_dout, coef, am, pwv, pb, s);
  launch(k_deform_bwd_reduce, dim3(static_cast<unsigned>(C + 1)), dim3(kBlock), 0, s, static_cast<const float*>(pwv),
         static_cast<const float*>(pb), static_cast<int64_t>(grid), C, dwv, dbeta);
  const int q = chunks <= lpr ? 1 : 2;
  const int64_t span_len = static_cast<int64_t>(kBlock / lpr) * chunk;
  const int64_t nspans = (total + span_len - 1) / span_len;
  deform_grad_dispatch(lpr, q, offsets, entries, chunk_first, chunk, n, total, dout, ld_dout, coef, am, wv, C, dvals,
                       ld_dvals, parts, parts + nspans * C, parts + 2 * nspans * C, s);
}

void launch_deform_slice(const int32_t* idx, const float* w, int64_t m, const void* vals,
                         int64_t ld_vals, int C, int bf16, const float* wv, float beta, float* out,
                         float* delta, float* plain, hipStream_t s) {
  if (m <= 0) return;
  const int chunks = C / (bf16 ? 8 : 4);
  const int lpr = point_lanes_per_row(C, bf16 != 0);
  ScopedKernelTimer tm("deform_slice", s);
  const bool two = chunks > lpr;
  if (bf16) {
    if (two) deform_dispatch<true, 2>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, plain, s);
    else deform_dispatch<true, 1>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, plain, s);
  } else {
    if (two) deform_dispatch<false, 2>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, plain, s);
    else deform_dispatch<false, 1>(lpr, idx, w, m, vals, ld_vals, C, wv, beta, out, delta, plain, s);
  }
}

}  // namespace lat

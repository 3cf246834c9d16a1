// Lattice convolution on gfx950 matrix cores.
//
// out[v] = bias + sum_t in[nb(v,t)] W[t]^T is a GEMM whose A operand is
// gathered: row v of A is the concatenation over the 9 taps of the input
// rows of v's neighbours (a zero row where the neighbour is missing).  The
// neighbour table is tap-major (nb[t][v]) so a wave reads the indices of its
// rows with one coalesced load per tap.  The same kernel runs the 1-hop
// convolution, the strided convolution of Downsample and the transposed
// convolution of Upsample; only the table differs.
//
// Each wave owns a (16 RM) x (16 RN) output tile in MFMA accumulators and
// walks K = 9 * Cin.  Operands go straight from global memory (L2) into
// registers in the MFMA operand layout: every lane loads 16 contiguous bytes
// of one input row (A) and of one weight row (B, weights stored
// [tap][Cout][Cin] so that the K dimension is contiguous for both).
//   fp32: v_mfma_f32_16x16x4_f32, a float4 per lane feeds 4 MFMAs (K = 16
//         per step: lane group g holds channels 4g..4g+3).
//   bf16: v_mfma_f32_16x16x32_bf16, 8 bf16 per lane feed one MFMA (K = 32
//         per step: lane group g holds channels 8g..8g+7).
// Any assignment of K indices to (lane group, element) works as long as A
// and B use the same one; the accumulator layout is fixed by the hardware:
// lane l holds rows 4*(l/16) + r, r = 0..3, of column l%16.
#include "lattice_internal.h"

namespace lat {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWaves = 4;
constexpr int kBlock = 64 * kWaves;

__device__ inline uint16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Operand fragment of one lane: 16 bytes of one row (A) or weight row (B).
template <bool BF16> struct Frag;
template <> struct Frag<false> {
  float4 v;
  __device__ inline void zero() { v = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ inline void load(const void* base, int64_t elem) {
    v = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
  }
};
template <> struct Frag<true> {
  u32x4 v;
  __device__ inline void zero() { v = u32x4{0u, 0u, 0u, 0u}; }
  __device__ inline void load(const void* base, int64_t elem) {
    v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + elem);
  }
};

__device__ inline void mma(f32x4& acc, const Frag<false>& a, const Frag<false>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.x, b.v.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.y, b.v.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.z, b.v.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v.w, b.v.w, acc, 0, 0, 0);
}
__device__ inline void mma(f32x4& acc, const Frag<true>& a, const Frag<true>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a.v), __builtin_bit_cast(bf16x8, b.v),
                                                 acc, 0, 0, 0);
}

// Workgroup of WM x WN waves; each wave owns (16 RM) x (16 RN) outputs.
template <bool BF16, int RM, int RN, int WM, int WN>
__global__ void __launch_bounds__(kBlock)
k_conv(const int32_t* __restrict__ nbr, int64_t ldn, int64_t n_out, const void* __restrict__ in,
       int64_t ld_in, int Cin, const void* __restrict__ W, const float* __restrict__ bias, int Cout,
       int relu, void* __restrict__ out, int64_t ld_out) {
  static_assert(WM * WN == kWaves, "four waves per workgroup");
  constexpr int KS = BF16 ? 32 : 16;          // channels per K step
  constexpr int EPL = BF16 ? 8 : 4;           // elements per lane per step
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int li = lane & 15;                   // row (A) / column (B) within a 16-block
  const int lg = lane >> 4;                   // K group
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * WM + wave % WM) * (16 * RM);
  const int col0 = (blockIdx.y * WN + wave / WM) * (16 * RN);

  f32x4 acc[RM][RN];
#pragma unroll
  for (int a = 0; a < RM; ++a)
#pragma unroll
    for (int b = 0; b < RN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // neighbour rows of every tap, loaded once
  int32_t nb[kTaps][RM];
#pragma unroll
  for (int t = 0; t < kTaps; ++t)
#pragma unroll
    for (int a = 0; a < RM; ++a) {
      const int64_t r = row0 + a * 16 + li;
      nb[t][a] = r < n_out ? nbr[t * ldn + r] : -1;
    }
  int64_t wrow[RN];
  bool col_ok[RN];
#pragma unroll
  for (int b = 0; b < RN; ++b) {
    const int col = col0 + b * 16 + li;
    col_ok[b] = col < Cout;
    wrow[b] = static_cast<int64_t>(col) * Cin;
  }
  const int64_t wtap = static_cast<int64_t>(Cout) * Cin;

  Frag<BF16> A[RM], B[RN], An[RM], Bn[RN];
  auto load = [&](int t, int c0, Frag<BF16>(&fa)[RM], Frag<BF16>(&fb)[RN]) {
    const int ch = c0 + lg * EPL;
    const bool k_ok = ch < Cin;
#pragma unroll
    for (int a = 0; a < RM; ++a) {
      if (k_ok && nb[t][a] >= 0) fa[a].load(in, static_cast<int64_t>(nb[t][a]) * ld_in + ch);
      else fa[a].zero();
    }
#pragma unroll
    for (int b = 0; b < RN; ++b) {
      if (k_ok && col_ok[b]) fb[b].load(W, t * wtap + wrow[b] + ch);
      else fb[b].zero();
    }
  };

  load(0, 0, A, B);
#pragma unroll
  for (int t = 0; t < kTaps; ++t) {
    for (int c0 = 0; c0 < Cin; c0 += KS) {
      // prefetch the next K step (next channels of this tap, or the next tap)
      if (c0 + KS < Cin) load(t, c0 + KS, An, Bn);
      else if (t + 1 < kTaps) load(t + 1, 0, An, Bn);
#pragma unroll
      for (int a = 0; a < RM; ++a)
#pragma unroll
        for (int b = 0; b < RN; ++b) mma(acc[a][b], A[a], B[b]);
#pragma unroll
      for (int a = 0; a < RM; ++a) A[a] = An[a];
#pragma unroll
      for (int b = 0; b < RN; ++b) B[b] = Bn[b];
    }
  }

  // epilogue: bias, ReLU, convert, store
#pragma unroll
  for (int b = 0; b < RN; ++b) {
    const int col = col0 + b * 16 + li;
    if (col >= Cout) continue;
    const float bb = bias ? bias[col] : 0.f;
#pragma unroll
    for (int a = 0; a < RM; ++a)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = row0 + a * 16 + lg * 4 + r;
        if (row >= n_out) continue;
        float v = acc[a][b][r] + bb;
        if (relu) v = fmaxf(v, 0.f);
        if constexpr (BF16)
          static_cast<uint16_t*>(out)[row * ld_out + col] = f32_to_bf16(v);
        else
          static_cast<float*>(out)[row * ld_out + col] = v;
      }
  }
}

template <bool BF16, int RM, int RN, int WM, int WN>
void conv_launch(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int relu, void* out,
                 int64_t ld_out, hipStream_t s) {
  const int64_t rows_per_block = static_cast<int64_t>(WM) * 16 * RM;
  const int cols_per_block = WN * 16 * RN;
  const dim3 grid(static_cast<unsigned>((n_out + rows_per_block - 1) / rows_per_block),
                  static_cast<unsigned>((Cout + cols_per_block - 1) / cols_per_block));
  hipLaunchKernelGGL((k_conv<BF16, RM, RN, WM, WN>), grid, dim3(kBlock), 0, s, nbr, ldn, n_out, in,
                     ld_in, Cin, W, bias, Cout, relu, out, ld_out);
}

int64_t blocks_of(int64_t n_out, int Cout, int rows, int cols) {
  return ((n_out + rows - 1) / rows) * ((Cout + cols - 1) / cols);
}

// Tile choice: the largest tile that still gives every CU a couple of
// workgroups; small lattice levels fall back to 16-row wave tiles.
template <bool BF16>
void conv_dispatch(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                   int Cin, const void* W, const float* bias, int Cout, int relu, void* out,
                   int64_t ld_out, hipStream_t s) {
  constexpr int64_t kWant = 512;
  if (Cout > 32 && blocks_of(n_out, Cout, 128, 64) >= kWant)
    return conv_launch<BF16, 2, 4, 4, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  if (Cout > 32 && blocks_of(n_out, Cout, 64, 64) >= kWant)
    return conv_launch<BF16, 1, 4, 4, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  if (Cout > 16)
    return conv_launch<BF16, 1, 2, 4, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  return conv_launch<BF16, 1, 1, 4, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
}

}  // namespace

void launch_conv(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int bf16, int relu, void* out,
                 int64_t ld_out, hipStream_t s) {
  if (n_out <= 0) return;
  ScopedKernelTimer tm("conv", s);
  if (bf16) conv_dispatch<true>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  else conv_dispatch<false>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
}

}  // namespace lat

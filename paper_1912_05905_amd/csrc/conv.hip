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

template <bool BF16, int RM, int RN>
__global__ void __launch_bounds__(kBlock)
k_conv(const int32_t* __restrict__ nbr, int64_t ldn, int64_t n_out, const void* __restrict__ in,
       int64_t ld_in, int Cin, const void* __restrict__ W, const float* __restrict__ bias, int Cout,
       int relu, void* __restrict__ out, int64_t ld_out) {
  constexpr int KS = BF16 ? 32 : 16;          // channels per K step
  constexpr int EPL = BF16 ? 8 : 4;           // elements per lane per step
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int li = lane & 15;                   // row (A) / column (B) within a 16-block
  const int lg = lane >> 4;                   // K group
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * kWaves + wave) * (16 * RM);
  const int col0 = blockIdx.y * (16 * RN);

  f32x4 acc[RM][RN];
#pragma unroll
  for (int a = 0; a < RM; ++a)
#pragma unroll
    for (int b = 0; b < RN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  bool col_ok[RN];
#pragma unroll
  for (int b = 0; b < RN; ++b) col_ok[b] = col0 + b * 16 + li < Cout;

  for (int t = 0; t < kTaps; ++t) {
    int32_t nb[RM];
#pragma unroll
    for (int a = 0; a < RM; ++a) {
      const int64_t r = row0 + a * 16 + li;
      nb[a] = r < n_out ? nbr[t * ldn + r] : -1;
    }
    for (int c0 = 0; c0 < Cin; c0 += KS) {
      const int ch = c0 + lg * EPL;
      const bool k_ok = ch < Cin;
      if constexpr (!BF16) {
        float4 av[RM], bv[RN];
#pragma unroll
        for (int a = 0; a < RM; ++a) {
          av[a] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (k_ok && nb[a] >= 0)
            av[a] = *reinterpret_cast<const float4*>(static_cast<const float*>(in) + nb[a] * ld_in + ch);
        }
#pragma unroll
        for (int b = 0; b < RN; ++b) {
          bv[b] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (k_ok && col_ok[b])
            bv[b] = *reinterpret_cast<const float4*>(
                static_cast<const float*>(W) + (static_cast<int64_t>(t) * Cout + col0 + b * 16 + li) * Cin + ch);
        }
#pragma unroll
        for (int a = 0; a < RM; ++a)
#pragma unroll
          for (int b = 0; b < RN; ++b) {
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a].x, bv[b].x, acc[a][b], 0, 0, 0);
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a].y, bv[b].y, acc[a][b], 0, 0, 0);
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a].z, bv[b].z, acc[a][b], 0, 0, 0);
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a].w, bv[b].w, acc[a][b], 0, 0, 0);
          }
      } else {
        u32x4 av[RM], bv[RN];
#pragma unroll
        for (int a = 0; a < RM; ++a) {
          av[a] = u32x4{0u, 0u, 0u, 0u};
          if (k_ok && nb[a] >= 0)
            av[a] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(in) + nb[a] * ld_in + ch);
        }
#pragma unroll
        for (int b = 0; b < RN; ++b) {
          bv[b] = u32x4{0u, 0u, 0u, 0u};
          if (k_ok && col_ok[b])
            bv[b] = *reinterpret_cast<const u32x4*>(
                static_cast<const uint16_t*>(W) + (static_cast<int64_t>(t) * Cout + col0 + b * 16 + li) * Cin + ch);
        }
#pragma unroll
        for (int a = 0; a < RM; ++a)
#pragma unroll
          for (int b = 0; b < RN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av[a]),
                                                                 __builtin_bit_cast(bf16x8, bv[b]),
                                                                 acc[a][b], 0, 0, 0);
      }
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

template <bool BF16, int RM, int RN>
void conv_launch(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int relu, void* out,
                 int64_t ld_out, hipStream_t s) {
  const int64_t rows_per_block = static_cast<int64_t>(kWaves) * 16 * RM;
  const dim3 grid(static_cast<unsigned>((n_out + rows_per_block - 1) / rows_per_block),
                  static_cast<unsigned>((Cout + 16 * RN - 1) / (16 * RN)));
  hipLaunchKernelGGL((k_conv<BF16, RM, RN>), grid, dim3(kBlock), 0, s, nbr, ldn, n_out, in, ld_in,
                     Cin, W, bias, Cout, relu, out, ld_out);
}

}  // namespace

void launch_conv(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int bf16, int relu, void* out,
                 int64_t ld_out, hipStream_t s) {
  if (n_out <= 0) return;
  ScopedKernelTimer tm("conv", s);
  if (bf16) {
    if (Cout <= 16) conv_launch<true, 2, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
    else if (Cout <= 32) conv_launch<true, 2, 2>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
    else conv_launch<true, 2, 4>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  } else {
    if (Cout <= 16) conv_launch<false, 2, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
    else if (Cout <= 32) conv_launch<false, 2, 2>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
    else conv_launch<false, 2, 4>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, s);
  }
}

}  // namespace lat

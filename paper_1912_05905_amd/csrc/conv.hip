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
#include <algorithm>
#include <type_traits>
#include <utility>

#include "lattice_internal.h"

namespace lat {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWaves = 4;
constexpr int kBlock = 64 * kWaves;

// Buffer resource word 3 for raw (untyped) buffer loads on CDNA, and an
// offset beyond any buffer the kernels build (at most kMaxBufferBytes), for
// which a buffer load returns zeros without a memory access.
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kMaxPreChannels = 1024;   // widest input of a pre-activated convolution
constexpr int kOutOfRange = static_cast<int>(0x80000000u);
constexpr int64_t kMaxBufferBytes = (int64_t{1} << 31) - 64;

// f(std::integral_constant<int, i>) for i = 0 .. N-1, unrolled.
template <class F, int... I>
__device__ inline void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ inline void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
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
       int relu, void* __restrict__ out, int64_t ld_out, const int32_t* __restrict__ rows) {
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
      nb[t][a] = r < n_out ? nbr[t * ldn + (rows ? rows[r] : r)] : -1;
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
        const int64_t r0 = row0 + a * 16 + lg * 4 + r;
        if (r0 >= n_out) continue;
        const int64_t row = rows ? rows[r0] : r0;
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
                 int64_t ld_out, const int32_t* rows, hipStream_t s) {
  const int64_t rows_per_block = static_cast<int64_t>(WM) * 16 * RM;
  const int cols_per_block = WN * 16 * RN;
  const dim3 grid(static_cast<unsigned>((n_out + rows_per_block - 1) / rows_per_block),
                  static_cast<unsigned>((Cout + cols_per_block - 1) / cols_per_block));
  launch((k_conv<BF16, RM, RN, WM, WN>), grid, dim3(kBlock), 0, s, nbr, ldn, n_out, in,
                     ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows);
}

// ---------------------------------------------------------------------------
// LDS-staged pipeline.  A stage is one tap and KC channels.  The whole
// workgroup gathers the stage's A tile (BM neighbour rows, KC channels) and
// B tile (BN weight rows, KC channels) into LDS with 16-byte loads, 8 or 16
// lanes per row segment; the next stage's global loads are issued before the
// current stage is multiplied, so their latency hides behind the MFMAs.  The
// 16-byte chunks of an LDS row are stored in an order permuted by the row
// (chunk c of row r at c ^ swz(r)), so that the 16 rows an MFMA fragment
// reads, and the chunks a copy writes, fall in different banks: measured on
// gfx950 with rocprofv3 (SQ_LDS_BANK_CONFLICT), rows padded by 16 bytes cost
// about 3 conflict cycles per ds_read_b128, these permutations none.
// Workgroups are numbered so that each XCD gets a contiguous range of row
// tiles: neighbouring rows (the gather's halo) then stay in that XCD's L2.
// ---------------------------------------------------------------------------
template <bool BF16, int BM, int BN, int WM, int WN, int KCB>
struct LdsConv {
  static constexpr int U = BF16 ? 2 : 4;            // bytes per element
  static constexpr int EPC = 16 / U;                // elements per 16-byte chunk
  static constexpr int KC = KCB / U;                // channels per stage
  static constexpr int CPR = KCB / 16;              // chunks per row per stage
  static constexpr int LDR = KC;                    // LDS row (elements), chunks permuted by swz
  // chunk permutation of row r: 4 chunks by (r / 2) mod 4, 8 or 16 chunks by r
  __device__ static inline int swz(int r) { return CPR == 4 ? (r >> 1) & 3 : r & (CPR - 1); }
  // element offset of channel chunk c of row r
  __device__ static inline int at(int r, int c) { return r * LDR + ((c ^ swz(r)) & (CPR - 1)) * EPC; }
  static constexpr int RM = BM / (16 * WM);
  static constexpr int RN = BN / (16 * WN);
  static constexpr int KS = BF16 ? 32 : 16;         // channels per MFMA step
  static constexpr int EPL = BF16 ? 8 : 4;          // elements per lane per MFMA step
  static constexpr int A_PER_T = BM * CPR / kBlock; // A chunks copied per thread
  static constexpr int B_PER_T = (BN * CPR + kBlock - 1) / kBlock;
  static constexpr int A_BYTES = BM * LDR * U;
  static constexpr int B_BYTES = BN * LDR * U;
  static constexpr int LDS_BYTES = 2 * (A_BYTES + B_BYTES) + kTaps * BM * 4 + 32 * 4;
  static_assert(WM * WN == kWaves, "four waves");
  static_assert(RM >= 1 && RN >= 1, "wave tile");
  static_assert(A_PER_T >= 1 && BM * CPR % kBlock == 0, "A copy split");
  static_assert(CPR == 4 || CPR == 8 || CPR == 16, "chunk permutation");
  static_assert(KC % KS == 0 && KS * U == 64, "an MFMA step reads 4 chunks of a row");
};

// PRE: the pre-activation of the input (Group Normalization folded into a
// per-channel scale and shift, then a ReLU) is applied to every gathered
// input value of a neighbour that exists, as the stage is copied to LDS;
// pre holds Cin scales then Cin shifts.
template <bool BF16, int BM, int BN, int WM, int WN, int KCB, int NS, bool BUF, int SCHED, bool PRE>
__global__ void __launch_bounds__(kBlock)
k_conv_lds(const int32_t* __restrict__ nbr, int64_t ldn, int64_t n_out, const void* __restrict__ in,
           int64_t ld_in, int Cin, const void* __restrict__ W, const float* __restrict__ bias, int Cout,
           int relu, void* __restrict__ out, int64_t ld_out, const int32_t* __restrict__ rows,
           unsigned row_tiles, int splits, float* __restrict__ part, uint32_t in_bytes, uint32_t w_bytes,
           const float* __restrict__ pre, const void* __restrict__ res, int64_t ld_res) {
  using P = LdsConv<BF16, BM, BN, WM, WN, KCB>;
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  E* As = reinterpret_cast<E*>(smem);
  E* Bs = reinterpret_cast<E*>(smem + 2 * P::A_BYTES);
  int32_t* nbt = reinterpret_cast<int32_t*>(smem + 2 * (P::A_BYTES + P::B_BYTES));
  int32_t* tflag = nbt + kTaps * BM;  // [16] tap used by some row of the tile
  int32_t* tlist = tflag + 16;        // [16] bf16: used taps, count in tlist[15]
  float* pre_s = reinterpret_cast<float*>(smem + P::LDS_BYTES);   // PRE: [Cin] scales, [Cin] shifts

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int li = lane & 15;
  const int lg = lane >> 4;
  // XCD-aware tile order: workgroup b runs on XCD b % 8; give each XCD a
  // contiguous range of (row tile, column tile) items, column tiles of a row
  // tile adjacent, so that the workgroups gathering the same input rows run
  // at the same time on one XCD and share its L2.
  const unsigned b = blockIdx.x;
  const unsigned col_tiles = (Cout + BN - 1) / BN;
  const unsigned items = row_tiles * col_tiles;
  const unsigned per_xcd = (items + 7) / 8;
  const unsigned item = (b % 8) * per_xcd + b / 8;
  if (item >= items) return;
  const unsigned tile = item / col_tiles;
  const int64_t row0 = static_cast<int64_t>(tile) * BM;
  const int col0 = static_cast<int>(item - tile * col_tiles) * BN;
  const int wm = wave % WM, wn = wave / WM;

  // split z of the K dimension takes taps [tb, te)
  const int tb = static_cast<int>(blockIdx.z) * kTaps / splits;
  const int te = (static_cast<int>(blockIdx.z) + 1) * kTaps / splits;
  // Taps that no row of the tile uses are skipped: their A rows are all
  // zero.  Rows are multiplied independently, so the result of a row does
  // not depend on which other rows share its tile.
  if (tid < 16) tflag[tid] = 0;
  if constexpr (PRE)
    for (int i = tid; i < 2 * Cin; i += kBlock) pre_s[i] = pre[i];
  __syncthreads();
  for (int i = tid; i < (te - tb) * BM; i += kBlock) {
    const int t = i / BM, r = i - t * BM;
    int32_t nb = -1;
    if (row0 + r < n_out) nb = nbr[(tb + t) * ldn + (rows ? rows[row0 + r] : row0 + r)];
    nbt[i] = nb;
    if (nb >= 0) tflag[t] = 1;
  }
  __syncthreads();
  // The used taps in order.  fp32: every thread packs them itself, 4 bits
  // each (no serial list, one barrier fewer).  bf16: one thread lists them
  // in LDS; the packed form costs the 128 x 128 tile enough registers to
  // lose a wave per SIMD.
  uint64_t tpack = 0;
  int ntaps = 0;
  if constexpr (BF16) {
    if (tid == 0) {
      int k = 0;
      for (int t = 0; t < te - tb; ++t)
        if (tflag[t]) tlist[k++] = t;
      tlist[15] = k;
    }
    __syncthreads();
    ntaps = tlist[15];
  } else {
#pragma unroll
    for (int t = 0; t < kTaps; ++t)
      if (t < te - tb && tflag[t]) {
        tpack |= static_cast<uint64_t>(t) << (4 * ntaps);
        ++ntaps;
      }
    // the same for every thread: keep it in scalar registers
    tpack = (static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(tpack >> 32))) << 32) |
            static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(tpack)));
    ntaps = __builtin_amdgcn_readfirstlane(ntaps);
  }
  auto tap_at = [&](int ti) {
    if constexpr (BF16) return static_cast<int>(tlist[ti]);
    else return static_cast<int>((tpack >> (4 * ti)) & 15);
  };

  const int kc_steps = (Cin + P::KC - 1) / P::KC;
  const int stages = ntaps * kc_steps;

  // global -> register copies of one stage.  Every load is issued, also for
  // a missing neighbour, a channel past Cin or a stage past the last: with
  // buffer loads (BUF) such a load gets an offset beyond the buffer and
  // reads zeros without touching memory; otherwise it reads a valid address
  // and the value is replaced by zeros.  With no load skipped, the number of
  // loads in flight is known, and the wait before a stage is copied to LDS
  // covers that stage's loads only, not the ones issued after it.
  using V = uint4;
  V ra[NS][P::A_PER_T], rb[NS][P::B_PER_T];
  // (unused without BUF, where the byte counts are 0)
  const __amdgpu_buffer_rsrc_t rin =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(in), 0, static_cast<int>(in_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rw =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(W), 0, static_cast<int>(w_bytes), kRsrcWord3);
  auto load16 = [&](const __amdgpu_buffer_rsrc_t& rs, const void* base, int64_t elem, bool ok) -> V {
    if constexpr (BUF) {
      const int off = ok ? static_cast<int>(elem * static_cast<int64_t>(sizeof(E))) : kOutOfRange;
      return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    } else {
      const V x = *reinterpret_cast<const V*>(static_cast<const E*>(base) + (ok ? elem : 0));
      return ok ? x : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto fetch = [&](auto set_c, int st) {
    constexpr int set = decltype(set_c)::value;
    const bool live = st < stages;
    const int ti = min(st / kc_steps, 15);
    const int t = live ? tap_at(ti) : 0;
    const int kc = (st - ti * kc_steps) * P::KC;
#pragma unroll
    for (int j = 0; j < P::A_PER_T; ++j) {
      const int q = tid + j * kBlock;
      const int r = q / P::CPR, cc = q % P::CPR;
      const int ch = kc + cc * P::EPC;
      const int32_t nb = nbt[t * BM + r];
      ra[set][j] = load16(rin, in, static_cast<int64_t>(nb) * ld_in + ch, live && nb >= 0 && ch < Cin);
    }
#pragma unroll
    for (int j = 0; j < P::B_PER_T; ++j) {
      const int q = tid + j * kBlock;
      const int r = q / P::CPR, cc = q % P::CPR;
      const int ch = kc + cc * P::EPC;
      const int col = col0 + r;
      rb[set][j] = load16(rw, W, (static_cast<int64_t>(tb + t) * Cout + col) * Cin + ch,
                          live && q < BN * P::CPR && col < Cout && ch < Cin);
    }
  };
  // stage st's copy from its register set to LDS buffer buf
  auto stash = [&](auto set_c, int buf, int st) {
    constexpr int set = decltype(set_c)::value;
    E* a = As + buf * (BM * P::LDR);
    E* bb = Bs + buf * (BN * P::LDR);
    int t = 0, kc = 0;
    if constexpr (PRE) {
      const int ti = min(st / kc_steps, 15);
      t = st < stages ? tap_at(ti) : 0;
      kc = (st - ti * kc_steps) * P::KC;
    }
#pragma unroll
    for (int j = 0; j < P::A_PER_T; ++j) {
      const int q = tid + j * kBlock;
      const int r = q / P::CPR, cc = q % P::CPR;
      V v = ra[set][j];
      if constexpr (PRE) {
        const int ch = kc + cc * P::EPC;
        if (st < stages && nbt[t * BM + r] >= 0 && ch < Cin) {
          uint32_t w[4] = {v.x, v.y, v.z, v.w};
          if constexpr (BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float lo = fmaxf(fmaf(__uint_as_float(w[i] << 16), pre_s[ch + 2 * i], pre_s[Cin + ch + 2 * i]), 0.f);
              const float hi = fmaxf(fmaf(__uint_as_float(w[i] & 0xffff0000u), pre_s[ch + 2 * i + 1],
                                          pre_s[Cin + ch + 2 * i + 1]), 0.f);
              w[i] = pack_bf16x2(lo, hi);
            }
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              w[i] = __float_as_uint(fmaxf(fmaf(__uint_as_float(w[i]), pre_s[ch + i], pre_s[Cin + ch + i]), 0.f));
          }
          v = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
      *reinterpret_cast<V*>(a + P::at(r, cc)) = v;
    }
#pragma unroll
    for (int j = 0; j < P::B_PER_T; ++j) {
      const int q = tid + j * kBlock;
      if (q < BN * P::CPR) {
        const int r = q / P::CPR, cc = q % P::CPR;
        *reinterpret_cast<V*>(bb + P::at(r, cc)) = rb[set][j];
      }
    }
  };

  f32x4 acc[P::RM][P::RN];
#pragma unroll
  for (int a = 0; a < P::RM; ++a)
#pragma unroll
    for (int c = 0; c < P::RN; ++c) acc[a][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  // NS stages of global loads in flight: stage st is multiplied from LDS
  // buffer st & 1 while stages st+1 .. st+NS-1 wait in register sets
  // (st+i) % NS.  After the multiply, stage st+1 goes to the other LDS
  // buffer and stage st+NS is loaded into the set that stage st vacated, so
  // a load has NS-1 steps to arrive.  Set indices are compile-time constants
  // so that the register sets stay in registers.
  static_for<NS>([&](auto i_c) { fetch(i_c, decltype(i_c)::value); });
  stash(std::integral_constant<int, 0>{}, 0, 0);
  __syncthreads();
  // One pipeline step: stage st is multiplied from LDS buffer st & 1; stage
  // st+1 goes from its register set to the other buffer and stage st+NS is
  // loaded into the set stage st vacated.  With SCHED 1 the copy and the
  // loads come first, so that they overlap the multiply.  All fragments of
  // the stage are read from LDS before the first MFMA.
  auto step = [&](auto set_c, int st) {
    constexpr int SET = decltype(set_c)::value;
    constexpr int NEXT = (SET + 1) % NS;
    const int buf = st & 1;
    if constexpr (SCHED == 1) {
      stash(std::integral_constant<int, NEXT>{}, buf ^ 1, st + 1);
      fetch(set_c, st + NS);
    }
    // rows of a fragment are 16-aligned blocks plus li, so the permutation
    // of the lane's row is that of li: MFMA step k reads chunk 4 k + lg
    const E* a = As + buf * (BM * P::LDR) + (wm * P::RM * 16 + li) * P::LDR;
    const E* bb = Bs + buf * (BN * P::LDR) + (wn * P::RN * 16 + li) * P::LDR;
    const int sw = P::swz(li);
    constexpr int NK = P::KC / P::KS;
    Frag<BF16> fa[NK][P::RM], fb[NK][P::RN];
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      const int ck = (((4 * k + lg) ^ sw) & (P::CPR - 1)) * P::EPC;
#pragma unroll
      for (int i = 0; i < P::RM; ++i) fa[k][i].load(a, i * 16 * P::LDR + ck);
#pragma unroll
      for (int j = 0; j < P::RN; ++j) fb[k][j].load(bb, j * 16 * P::LDR + ck);
    }
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < P::RM; ++i)
#pragma unroll
          for (int j = 0; j < P::RN; ++j) mma(acc[i][j], fa[k][i], fb[k][j]);
      } else {
        // interleave independent accumulators between dependent MFMAs
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < P::RM; ++i)
#pragma unroll
            for (int j = 0; j < P::RN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[k][i].v[e], fb[k][j].v[e], acc[i][j], 0, 0, 0);
      }
    }
    if constexpr (SCHED == 0) {
      // unconditional: past the last stage these copy and load zeros
      stash(std::integral_constant<int, NEXT>{}, buf ^ 1, st + 1);
      fetch(set_c, st + NS);
    }
    __syncthreads();
  };
  // whole groups of NS steps without branches, then the remaining steps
  int st = 0;
  for (; st + NS <= stages; st += NS)
    static_for<NS>([&](auto i_c) { step(i_c, st + decltype(i_c)::value); });
  static_for<NS>([&](auto i_c) {
    if (st + decltype(i_c)::value < stages) step(i_c, st + decltype(i_c)::value);
  });

  if (part) {
    // raw partial sums of this split, [split][n_out][Cout]
    float* dst = part + static_cast<int64_t>(blockIdx.z) * n_out * Cout;
#pragma unroll
    for (int j = 0; j < P::RN; ++j) {
      const int col = col0 + (wn * P::RN + j) * 16 + li;
      if (col >= Cout) continue;
#pragma unroll
      for (int i = 0; i < P::RM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = row0 + (wm * P::RM + i) * 16 + lg * 4 + r;
          if (row < n_out) dst[row * Cout + col] = acc[i][j][r];
        }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < P::RN; ++j) {
    const int col = col0 + (wn * P::RN + j) * 16 + li;
    if (col >= Cout) continue;
    const float bv = bias ? bias[col] : 0.f;
#pragma unroll
    for (int i = 0; i < P::RM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t r0 = row0 + (wm * P::RM + i) * 16 + lg * 4 + r;
        if (r0 >= n_out) continue;
        const int64_t row = rows ? rows[r0] : r0;
        float v = acc[i][j][r] + bv;
        if (relu) v = fmaxf(v, 0.f);
        if constexpr (BF16) {
          if (res) v += __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(res)[row * ld_res + col]) << 16);
          static_cast<uint16_t*>(out)[row * ld_out + col] = f32_to_bf16(v);
        } else {
          if (res) v += static_cast<const float*>(res)[row * ld_res + col];
          static_cast<float*>(out)[row * ld_out + col] = v;
        }
      }
  }
}

// Sum of the split partials in split order, then bias, ReLU and conversion.
// Partial row r belongs to output row rows[r] when the tiles ran over a row
// order.
template <bool BF16>
__global__ void __launch_bounds__(kBlock)
k_conv_reduce(const float* __restrict__ part, int splits, int64_t n_out, int Cout, const float* __restrict__ bias,
              int relu, void* __restrict__ out, int64_t ld_out, const void* __restrict__ res, int64_t ld_res,
              const int32_t* __restrict__ rows) {
  const int64_t quads = n_out * (Cout / 4);
  const int64_t plane = n_out * Cout;
  for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < quads;
       q += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t prow = q / (Cout / 4);
    const int col = static_cast<int>(q - prow * (Cout / 4)) * 4;
    float4 a = *reinterpret_cast<const float4*>(part + prow * Cout + col);
    for (int z = 1; z < splits; ++z) {
      const float4 b = *reinterpret_cast<const float4*>(part + z * plane + prow * Cout + col);
      a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    }
    const int64_t row = rows ? rows[prow] : prow;
    float v[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (bias) v[i] += bias[col + i];
      if (relu) v[i] = fmaxf(v[i], 0.f);
      if (res) {
        if constexpr (BF16)
          v[i] += __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(res)[row * ld_res + col + i]) << 16);
        else
          v[i] += static_cast<const float*>(res)[row * ld_res + col + i];
      }
    }
    if constexpr (BF16) {
      const uint32_t lo = pack_bf16x2(v[0], v[1]);
      const uint32_t hi = pack_bf16x2(v[2], v[3]);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + row * ld_out + col) = make_uint2(lo, hi);
    } else {
      *reinterpret_cast<float4*>(static_cast<float*>(out) + row * ld_out + col) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// Byte extents of the gathered operands, for the buffer resources.
struct ConvExtent {
  int64_t in_bytes, w_bytes;
  bool buffer_ok() const { return in_bytes <= kMaxBufferBytes && w_bytes <= kMaxBufferBytes; }
};

template <bool BF16, int BM, int BN, int WM, int WN, int KCB, int NS = 2, bool BUF = true, int SCHED = 0,
          bool PRE = false>
void conv_lds_launch(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                     int Cin, const void* W, const float* bias, int Cout, int relu, void* out,
                     int64_t ld_out, const int32_t* rows, ConvExtent ext, hipStream_t s, const float* pre = nullptr,
                     const void* res = nullptr, int64_t ld_res = 0, int splits = 1, float* part = nullptr) {
  using P = LdsConv<BF16, BM, BN, WM, WN, KCB>;
  const int lds = P::LDS_BYTES + (PRE ? 8 * Cin : 0);
  static bool lds_limit_set = false;
  if (!lds_limit_set) {
    (void)hipFuncSetAttribute(
        reinterpret_cast<const void*>(&k_conv_lds<BF16, BM, BN, WM, WN, KCB, NS, BUF, SCHED, PRE>),
        hipFuncAttributeMaxDynamicSharedMemorySize, P::LDS_BYTES + (PRE ? 8 * kMaxPreChannels : 0));
    lds_limit_set = true;
  }
  const int64_t tiles = (n_out + BM - 1) / BM;
  const int64_t items = tiles * ((Cout + BN - 1) / BN);
  const unsigned per_xcd = static_cast<unsigned>((items + 7) / 8);
  const dim3 grid(per_xcd * 8, 1, static_cast<unsigned>(splits));
  launch((k_conv_lds<BF16, BM, BN, WM, WN, KCB, NS, BUF, SCHED, PRE>), grid, dim3(kBlock), static_cast<uint32_t>(lds),
         s, nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, static_cast<unsigned>(tiles),
         splits, splits > 1 ? part : nullptr, static_cast<uint32_t>(BUF ? ext.in_bytes : 0),
         static_cast<uint32_t>(BUF ? ext.w_bytes : 0), pre, res, ld_res);
  if (splits > 1) {
    const int64_t quads = n_out * (Cout / 4);
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((quads + kBlock - 1) / kBlock, 8192));
    launch((k_conv_reduce<BF16>), dim3(blocks), dim3(kBlock), 0, s, part, splits, n_out, Cout, bias,
                       relu, out, ld_out, res, ld_res, rows);
  }
}

int64_t blocks_of(int64_t n_out, int Cout, int rows, int cols) {
  return ((n_out + rows - 1) / rows) * ((Cout + cols - 1) / cols);
}

// Tile choice, from a sweep of tile shapes, pipeline depths and step
// schedules over the lattices of the LiDAR scan (fp32) and of the 1M-point
// room (bf16) on MI355X.  fp32: small tiles win; the levels are small and a
// stage costs several times its MFMA time.  Around a thousand 32 x 32 tiles
// a third stage in flight (with half the channels per stage) pays; a few
// hundred 32 x 64 tiles do best with two stages of 64 channels.  bf16: 128 x 128 tiles halve the
// gathered bytes per flop and win once there are enough of them (wide
// layers, large levels); 128 x 64 with stages of 32 channels for 64 output
// channels on large levels (half the weight rows per output row); 64 x 64
// otherwise.
// PRE (the pre-activated convolution) uses the same tiles, apart from the
// register kernel for narrow outputs, which has no pre-activation.
template <bool BF16, bool PRE>
void conv_dispatch(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* in, int64_t ld_in,
                   int Cin, const void* W, const float* bias, int Cout, int relu, void* out,
                   int64_t ld_out, const int32_t* rows, ConvExtent ext, hipStream_t s, const float* pre,
                   const void* res, int64_t ld_res) {
  if (!PRE && !res && Cout <= 16)
    return conv_launch<BF16, 1, 1, 4, 1>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, s);
  if (!ext.buffer_ok())  // operands beyond the reach of a buffer resource
    return conv_lds_launch<BF16, 64, 64, 2, 2, 128, 2, false, 0, PRE>(
        nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
  if constexpr (BF16) {
    const int64_t b128 = blocks_of(n_out, Cout, 128, 128);
    const int64_t b64 = blocks_of(n_out, Cout, 64, 64);
    if (Cout >= 128 && (b128 >= 1500 || (Cin >= 256 && Cout % 128 == 0)))
      return conv_lds_launch<true, 128, 128, 2, 2, 64, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (Cout == 64 && b64 >= 8192)
      return conv_lds_launch<true, 128, 64, 2, 2, 64, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (Cout > 32 && b64 >= 8192)
      return conv_lds_launch<true, 64, 64, 2, 2, 128, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (Cout > 32 && b64 >= 256)
      return conv_lds_launch<true, 64, 64, 2, 2, 128, 2, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    return conv_lds_launch<true, 32, 32, 2, 2, 128, 2, true, 0, PRE>(
        nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
  } else {
    if (Cout > 32 && blocks_of(n_out, Cout, 64, 64) >= 2048)
      return conv_lds_launch<false, 64, 64, 2, 2, 128, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (Cout > 64 && blocks_of(n_out, Cout, 32, 64) >= 1024)
      return conv_lds_launch<false, 32, 64, 2, 2, 128, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (Cout > 64 && blocks_of(n_out, Cout, 32, 64) >= 400)
      return conv_lds_launch<false, 32, 64, 2, 2, 256, 2, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    if (blocks_of(n_out, Cout, 32, 32) >= 1024)
      return conv_lds_launch<false, 32, 32, 2, 2, 128, 3, true, 1, PRE>(
          nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
    return conv_lds_launch<false, 32, 32, 2, 2, 256, 2, true, 1, PRE>(
        nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout, relu, out, ld_out, rows, ext, s, pre, res, ld_res);
  }
}

}  // namespace

int conv_max_pre_channels() { return kMaxPreChannels; }

void launch_conv(const int32_t* nbr, int64_t ldn, int64_t n_out, int64_t n_in, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int bf16, int relu, void* out,
                 int64_t ld_out, const int32_t* rows, hipStream_t s, const float* pre, const void* res,
                 int64_t ld_res) {
  if (n_out <= 0) return;
  ScopedKernelTimer tm("conv", s);
  const int64_t u = bf16 ? 2 : 4;
  const ConvExtent ext{n_in > 0 ? ((n_in - 1) * ld_in + Cin) * u : 0, int64_t{kTaps} * Cout * Cin * u};
  auto go = [&](auto bf_c, auto pre_c) {
    conv_dispatch<decltype(bf_c)::value, decltype(pre_c)::value>(nbr, ldn, n_out, in, ld_in, Cin, W, bias, Cout,
                                                                  relu, out, ld_out, rows, ext, s, pre, res, ld_res);
  };
  using T = std::true_type;
  using F = std::false_type;
  if (pre) bf16 ? go(T{}, T{}) : go(F{}, T{});
  else bf16 ? go(T{}, F{}) : go(F{}, F{});
}

}  // namespace lat

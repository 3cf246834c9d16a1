// Internal declarations of liblattice (gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "lattice.h"

namespace lat {

constexpr int kDim = 3;                 // d
constexpr int kVerts = kDim + 1;        // d+1 vertices per simplex, coordinates per key
constexpr int kTaps = 2 * kVerts + 1;   // 1-hop neighbourhood incl. the centre
constexpr int kMaskBins = 1 << kTaps;   // tap masks (bit t: tap t present)
constexpr int kCoordBits = 21;
constexpr int32_t kCoordLimit = 1 << 20;          // |c_i| < 2^20
constexpr uint64_t kEmptyKey = ~0ull;             // bit 63 set: never a packed key

// error bits raised by kernels into the handle's device flag
enum : uint32_t { kErrHashFull = 1u, kErrKeyRange = 2u, kErrNonFinite = 4u };

// Packed key: the first d coordinates, each biased by 2^20 into 21 bits
// (the last coordinate is minus their sum).  Unsigned order of packed keys is
// the lexicographic order of the coordinates.
__host__ __device__ inline bool coords_in_range(int32_t c0, int32_t c1, int32_t c2, int32_t c3) {
  return c0 > -kCoordLimit && c0 < kCoordLimit && c1 > -kCoordLimit && c1 < kCoordLimit &&
         c2 > -kCoordLimit && c2 < kCoordLimit && c3 > -kCoordLimit && c3 < kCoordLimit;
}

__host__ __device__ inline uint64_t pack_key(int32_t c0, int32_t c1, int32_t c2) {
  return (static_cast<uint64_t>(static_cast<uint32_t>(c0 + kCoordLimit)) << (2 * kCoordBits)) |
         (static_cast<uint64_t>(static_cast<uint32_t>(c1 + kCoordLimit)) << kCoordBits) |
         static_cast<uint64_t>(static_cast<uint32_t>(c2 + kCoordLimit));
}

__host__ __device__ inline void unpack_key(uint64_t k, int32_t c[kVerts]) {
  const uint64_t mask = (1ull << kCoordBits) - 1;
  c[0] = static_cast<int32_t>((k >> (2 * kCoordBits)) & mask) - kCoordLimit;
  c[1] = static_cast<int32_t>((k >> kCoordBits) & mask) - kCoordLimit;
  c[2] = static_cast<int32_t>(k & mask) - kCoordLimit;
  c[3] = -(c[0] + c[1] + c[2]);
}

// float32 -> bfloat16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
typedef __bf16 lat_bf16x2 __attribute__((ext_vector_type(2)));
typedef float lat_f32x2 __attribute__((ext_vector_type(2)));
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(lat_f32x2{lo, hi}, lat_bf16x2));
}
__device__ inline uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }

// Slot hash: the murmur3 64-bit finaliser.
__host__ __device__ inline uint64_t hash_key(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

// Open-addressing table with linear probing.  A slot is 16 bytes: the
// packed key (kEmptyKey when free), the vertex number and the number of
// point references of the vertex, so a probe reads one aligned 16-byte
// entry and the reference count shares the cache line the insert claimed.
struct alignas(16) HashEntry {
  uint64_t key;
  int32_t val;
  int32_t count;
};

struct HashView {
  HashEntry* e;
  uint64_t mask;      // capacity - 1 (capacity a power of two)
};

// Look up a key; -1 when absent.  The table is not modified concurrently.
__device__ inline int32_t hash_find(const HashView& h, uint64_t key) {
  uint64_t slot = hash_key(key) & h.mask;
  for (uint64_t probe = 0; probe <= h.mask; ++probe) {
    const uint4 ent = *reinterpret_cast<const uint4*>(&h.e[slot]);
    const uint64_t k = (static_cast<uint64_t>(ent.y) << 32) | ent.x;
    if (k == key) return static_cast<int32_t>(ent.z);
    if (k == kEmptyKey) return -1;
    slot = (slot + 1) & h.mask;
  }
  return -1;
}

// Key of lattice point c (d+1 coordinates), or kEmptyKey when c is out of
// range (such a point can never be a vertex).
__device__ inline uint64_t key_or_empty(const int32_t c[kVerts]) {
  return coords_in_range(c[0], c[1], c[2], c[3]) ? pack_key(c[0], c[1], c[2]) : kEmptyKey;
}

// Tap offsets o_t: 0; +n_j; -n_j with n_j = (d+1) e_j - 1.
__device__ inline int32_t tap_offset(int t, int i) {
  if (t == 0) return 0;
  const int j = (t - 1) & 3;
  const int32_t v = (i == j ? kVerts : 0) - 1;
  return t <= kVerts ? v : -v;
}

// ---------------------------------------------------------------------------
// host-side pieces shared by the translation units
// ---------------------------------------------------------------------------
struct Timer;   // kernel-family event timer (api.hip)
// Kernel-family timing: while a ScopedKernelTimer of an enabled family is
// alive on this thread, every launch() is bracketed by a start and a stop
// event (created without the system-scope fence), so the family's time is
// the sum of its kernels' execution times.  Scopes nest; the outermost one
// names the family (a backward operator that reuses a forward kernel is
// timed as the backward operator).
void timer_begin(const char* family);
void timer_end();
bool timer_take_events(hipEvent_t* start, hipEvent_t* stop);

struct ScopedKernelTimer {
  ScopedKernelTimer(const char* f, hipStream_t) { timer_begin(f); }
  ~ScopedKernelTimer() { timer_end(); }
};

// Timed launches bind their events to the kernel's own dispatch
// (hipExtLaunchKernel), so timing adds no marker packets between kernels.
template <typename K, typename... Args>
inline void launch(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (timer_take_events(&e0, &e1))
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, e0, e1, 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}

// A launch whose completion also completes `done` (bound to the dispatch;
// a separate event record only when the launch is timed as well).
template <typename K, typename... Args>
inline void launch_signal(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, hipEvent_t done,
                          Args... args) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (timer_take_events(&e0, &e1)) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, e0, e1, 0u, args...);
    (void)hipEventRecord(done, s);
  } else {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, static_cast<hipEvent_t>(nullptr), done, 0u, args...);
  }
}

// Build work batched over the levels of a hierarchy: tables cleared in one
// launch, tables' rows ordered by tap mask in one launch.
struct ClearJob {
  HashEntry* entries;
  int64_t cap;
  void* dev_counters;   // the level's device counters (zeroed)
  void* scan_work;      // the level's scan status words (zeroed)
};
constexpr int kMaxLevels = 8;   // levels of one hierarchy call (one launch job each)
// One level's insert.  The elevated positions come from `pos` (m x 3) with
// the factors a0..a2, then halved `halvings` times (a level that many steps
// coarser than the finest), or, without `pos`, from y_in times y_scale.
struct InsertJob {
  const float* pos;
  const float* y_in;
  float y_scale;
  int halvings;
  float a0, a1, a2;
  HashView h;
  int32_t* counter;
  uint64_t* vkeys;
  int32_t* vslot;
  int32_t* slot_out;
  int32_t* rank_out;
  float* w_out;
  float* y_out;
  uint32_t* err;
  int32_t* host_counts;
  uint32_t stamp;
};
// One level's convolution tables: the same-level table, and for a coarse
// level its Downsample table and the Upsample table into the finer level.
struct TableJob {
  HashView h;            // the level's hash table
  HashView hf;           // the finer level's (coarse levels)
  const uint64_t* keys;  // the level's vertex keys
  const uint64_t* fkeys; // the finer level's (coarse levels)
  const int32_t* n_dev;  // the level's vertex count (device)
  const int32_t* nf_dev; // the finer level's (coarse levels)
  int32_t* nbr;          // same-level table, tap-major, row stride ld
  int32_t* down;         // Downsample table, row stride ld (null for the finest level)
  int32_t* up;           // Upsample table, row stride ldf (null for the finest level)
  int64_t ld, ldf;
};
struct RowOrderJob {
  const int32_t* nbr;   // tap-major table, row stride ld
  int64_t ld;
  const int32_t* n_dev; // its row count (device)
  int32_t* rows;        // out: its rows grouped by tap mask within ranges
};
constexpr int kMaxRowOrderJobs = 8;
// Filled by launch_neighbor_table (one job) and launch_coarse_tables (three);
// the caller keeps n + jobs <= kMaxRowOrderJobs, launching the batch
// (launch_row_orders) when the next level would not fit.
struct RowOrderBatch {
  RowOrderJob job[kMaxRowOrderJobs];
  int n = 0;
  int64_t max_rows = 0;  // bound on the jobs' row counts (host)
  void add(const RowOrderJob& j, int64_t rows_max) {
    job[n++] = j;
    if (rows_max > max_rows) max_rows = rows_max;
  }
};

// Launchers (each .hip file implements its own kernels' launchers).
// create.hip
void launch_clear_table(HashEntry* entries, int64_t cap, void* dev_counters, void* scan_work,
                        hipStream_t s);
void launch_clear_tables(const ClearJob* jobs, int n, hipStream_t s);
// the inserts of n levels of one cloud of m points in one launch; done[i]
// is recorded once level i's insert has completed
void launch_insert_levels(const InsertJob* jobs, const hipEvent_t* done, int n, int64_t m, hipStream_t s);
int64_t scan_workspace_bytes();
void launch_count_scan(const HashEntry* table, const int32_t* vslot, const int32_t* n_dev,
                       int32_t* offsets, void* work, hipStream_t s);
void launch_fill_lists(HashView h, const int32_t* slot, const int32_t* rank, const float* w,
                       const int32_t* offsets, int32_t* idx, int32_t* entries, float* entry_w,
                       int32_t* chunk_first, int chunk, int64_t m4, hipStream_t s);
// the table, then its rows grouped by tap mask within ranges of 4096
// (nbr_rows); with `defer` the row order is added to that batch instead of
// launched
void launch_neighbor_table(HashView h, const uint64_t* vkeys, const int32_t* n_dev, int64_t n_max,
                           int32_t* nbr, int64_t ldn, int32_t* nbr_rows, hipStream_t s,
                           RowOrderBatch* defer = nullptr);
void launch_coarse_tables(HashView coarse, HashView fine, const uint64_t* coarse_keys, const uint64_t* fine_keys,
                          const int32_t* nc_dev, const int32_t* nf_dev, int64_t nc_max, int64_t nf_max, int32_t* nbr,
                          int32_t* down, int32_t* up, int32_t* up_rows, int32_t* nbr_rows, int32_t* down_rows,
                          hipEvent_t done, hipStream_t s, RowOrderBatch* defer = nullptr);
// the batch's row orders in one launch (`done`, if given, bound to it)
void launch_row_orders(const RowOrderBatch& b, hipEvent_t done, hipStream_t s);
// the tables of n levels in one launch (row orders not included); work_max
// bounds any job's (row, tap) entries
void launch_level_tables(const TableJob* jobs, int n, int64_t work_max, hipStream_t s);
void launch_export_keys(const uint64_t* vkeys, int64_t n, int32_t* out, hipStream_t s);
// adds to *count the (row, tap) pairs of the first n rows whose entry is >= 0
void launch_count_taps(const int32_t* tab, int64_t ld, int64_t n, unsigned long long* count, hipStream_t s);
void launch_transpose_table(const int32_t* tab, int64_t ld, int64_t n, int32_t* out, hipStream_t s);
// splat_slice.hip
int64_t splat_partial_floats(int64_t total, int chunk, int C);
void launch_splat(const int32_t* offsets, const int32_t* entries, const float* entry_w,
                  const int32_t* chunk_first, int chunk, int64_t n_max, int64_t total,
                  const void* feat, int64_t ld_feat, int C, int bf16, int normalize, void* vals,
                  int64_t ld_vals, float* wsum, float* partials, hipStream_t s);
void launch_slice(const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ld_vals,
                  int C, int bf16, float* out, hipStream_t s);
void launch_deform_slice(const int32_t* idx, const float* w, int64_t m, const void* vals,
                         int64_t ld_vals, int C, int bf16, const float* wv, float beta, float* out,
                         float* delta, float* plain, hipStream_t s);
int deform_classify_max_classes();
int deform_classify_max_weights();
void launch_deform_classify(const int32_t* idx, const float* w, int64_t m, const void* vals, int64_t ld_vals, int C,
                            int bf16, const float* wv, float beta, const float* Wc, const float* bc, int K, float* out,
                            hipStream_t s);
int64_t deform_backward_workspace_bytes(int64_t m, int C, int64_t total, int chunk);
void launch_deform_slice_backward(const int32_t* idx, const float* w, int64_t m, const int32_t* offsets,
                                  const int32_t* entries, const int32_t* chunk_first, int chunk, int64_t n,
                                  int64_t total, const float* vals, int64_t ld_vals, int C, const float* wv,
                                  float beta, const float* dout, int64_t ld_dout, float* dvals, int64_t ld_dvals,
                                  float* dwv, float* dbeta, void* work, hipStream_t s);
// distribute.hip
int64_t distribute_workspace_bytes(int64_t n, int64_t total, int C3, int out_bf16);
int distribute_max_features();
// scale: sigma per axis at the lattice's level (positions enter as pos / scale);
// gamma / beta: optional per-channel parameters of the three GroupNorms,
// concatenated ((3 + cf) + C1 + C2 values)
// Distribute + PointNet backward (dL/dx = dX, n x C3): dF (m x cf), the
// layers' dW ([out][in]) and db, dgamma / dbeta (concatenated as gamma); any
// output may be NULL.  work holds distribute_backward_workspace_bytes.
int64_t distribute_backward_workspace_bytes(int64_t n, int64_t m, int64_t total, int cf, int C1, int C2, int C3);
void launch_distribute_backward(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                                int64_t n, int64_t m, int64_t total, const float* pos, const double scale[3],
                                const float* feat, int64_t ld_feat, int cf, const float* gamma, const float* beta,
                                float eps, const float* W1, const float* b1, int C1, const float* W2, const float* b2,
                                int C2, const float* W3, const float* b3, int C3, const float* dX, int64_t ld_dX,
                                float* dF, int64_t ld_dF, float* dW1, float* db1, float* dW2, float* db2, float* dW3,
                                float* db3, float* dgamma, float* dbeta, void* work, hipStream_t s);
void launch_distribute(const int32_t* offsets, const int32_t* entries, const int32_t* chunk_first, int chunk,
                       int64_t n, int64_t total, const float* pos, const double scale[3], const float* feat,
                       int64_t ld_feat, int cf, const float* gamma, const float* beta, float eps, const float* W1,
                       const float* b1, int C1, const float* W2, const float* b2, int C2, const float* W3,
                       const float* b3, int C3, void* out, int out_bf16, int64_t ld_out, void* work, hipStream_t s);
// backward.hip
void launch_scale_by_weight_sum(const int32_t* offsets, const float* entry_w, const float* wsum, int64_t n,
                                const float* in, int64_t ld_in, int C, float* out, int64_t ld_out, hipStream_t s);
// dY, Y, G, W, Wt (and X below) are float32, or bfloat16 with bf16 != 0
void launch_conv_bwd_prep(const void* dY, int64_t ld_dy, const void* Y, int64_t ld_y, int64_t n, void* G,
                          int64_t ld_g, const void* W, int Cout, int Cin, void* Wt, int bf16, hipStream_t s);
int64_t wgrad_partial_floats(int64_t n_out, int Cout, int Cin);
void launch_conv_wgrad(const int32_t* nbr, int64_t ldn, int64_t n_out, const void* X, int64_t ld_x, int Cin,
                       const void* G, int64_t ld_g, int Cout, float* dW, float* dbias, float* partials, int bf16,
                       hipStream_t s);
// conv.hip
// pre: optional Cin scales then Cin shifts of the pre-activation (applied,
// with a ReLU, to the gathered input values of existing neighbours);
// res: optional residual (n_out x Cout, out's dtype) added after the
// activation of the output
void launch_conv(const int32_t* nbr, int64_t ldn, int64_t n_out, int64_t n_in, const void* in, int64_t ld_in,
                 int Cin, const void* W, const float* bias, int Cout, int bf16, int relu, void* out,
                 int64_t ld_out, const int32_t* rows, hipStream_t s, const float* pre = nullptr,
                 const void* res = nullptr, int64_t ld_res = 0);
int conv_max_pre_channels();
// norm.hip
int gn_max_channels();
int64_t gn_workspace_bytes(int64_t n, int C);
// stats (optional): per group the mean and 1 / sqrt(var + eps), as doubles
void launch_gn_affine(const void* x, int64_t ld, int C, int bf16, int64_t n, int groups, const float* gamma,
                      const float* beta, float eps, float* pre, void* work, hipStream_t s, double* stats = nullptr);
// classifier backward (z = dL/dlogits, m x K; f the DeformSlice output,
// m x C dense): df = z Wc (m x C dense), dWc = z^T f, dbc = column sums of
// z (either may be NULL); part holds classify_backward_partial_floats
int64_t classify_backward_partial_floats(int64_t m, int K, int C);
// backward of out_p = W a_p + b over m rows (W: K x C [out][in], dense, 16-byte
// aligned, C a multiple of 4) for z = dL/dout (m x K, row stride ld_z):
// df = z W (m x C, row stride ld_df; NULL: skipped), dW = z^T a written as
// K x C_out (the first C_out columns), db = column sums of z (either NULL:
// skipped).  a = f (row stride ld_f), or max(f scale + shift, 0) with pre =
// [C scales][C shifts].  part holds classify_backward_partial_floats(m, K, C).
void launch_linear_backward(const float* z, int64_t ld_z, const float* W, int K, int C, int64_t m, const float* f,
                            int64_t ld_f, const float* pre, float* df, int64_t ld_df, float* dW, int C_out, float* db,
                            float* part, hipStream_t s);
void launch_classify_backward(const float* z, int64_t ld_z, const float* Wc, int K, int C, int64_t m, const float* f,
                              float* df, float* dWc, float* dbc, float* part, hipStream_t s);
// a = max(x pre[c] + pre[C + c], 0) for fp32 x (n x C), the pre-activated
// input the convolution gathered
void launch_gn_relu_apply(const float* x, int64_t ldx, int C, int64_t n, const float* pre, float* a, int64_t lda,
                          hipStream_t s);
// GroupNorm + ReLU backward from dA = dL/d(pre-activated input): dgamma,
// dbeta (optional, C floats), dX (optional, n x C, row stride lddx); coef
// is a 4 C float work array; work holds gn_workspace_bytes(n, C).  The ReLU
// passed where act > 0 when the forward's activations act (n x C, row
// stride ldact) are given, else where x pre[c] + pre[C + c] > 0.  With
// xhat the rows x are given already normalised ((x - mean_g) inv_g).
void launch_gn_backward(const float* x, int64_t ldx, const float* dA, int64_t lda, int C, int groups, int64_t n,
                        const float* gamma, const float* pre, const double* stats, float* dgamma, float* dbeta,
                        float* coef, float* dX, int64_t lddx, void* work, hipStream_t s,
                        const float* act = nullptr, int64_t ldact = 0, bool xhat = false);
// per-group statistics from nparts partials (part[w][0..C) sums, part[w][C..2C)
// sums of squares over `rows` rows) -> pre[0..C) scales, pre[C..2C) shifts
void launch_gn_finalize(const double* part, int64_t nparts, int C, int groups, int64_t rows, const float* gamma,
                        const float* beta, float eps, float* pre, hipStream_t s, double* stats = nullptr);

}  // namespace lat

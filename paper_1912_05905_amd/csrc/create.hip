// Lattice construction on gfx950: point embedding, device hash insert,
// vertex numbering, per-vertex point lists J_v and the neighbour tables.
//
// The embedding (elevation, rounding, ranking, barycentric weights) must
// produce the vertex set bit for bit, so this file is compiled with float
// contraction off and every float operation below is one IEEE rounding.
//
// Device-scope atomics on this part are resolved beyond the per-XCD L2, so
// the insert kernel keeps them off the per-reference path: a workgroup first
// merges its 1024 vertex references in an LDS hash table, then touches the
// global table once per distinct key, adds its reference count for that key
// with one atomic, and numbers all vertices it created with one atomic on
// the vertex counter.  With one wave of workgroups the kernel's time is the
// latency of that chain, so a thread probes for all of its distinct keys at
// once (each probe a compare-and-swap, whose result also says whether the
// slot holds the key) and leaves its count atomics in flight while the
// workgroup numbers its new vertices.
#pragma clang fp contract(off)

#include <algorithm>

#include "lattice_internal.h"

namespace lat {
namespace {

constexpr int kBlock = 256;
constexpr int kLdsSlots = 2048;             // LDS table: 2x the references of a workgroup
constexpr int kLdsPerThread = kLdsSlots / kBlock;

// ---- exclusive scan of per-vertex counts over a device-side n ----
// kScanBlocks workgroups each own a contiguous range of vertices (the count
// of vertex v is table[vslot[v]].count).  Single pass: a workgroup publishes
// the sum of its range in scan_status, adds the published sums of the
// earlier ranges and scans its own range.
constexpr int kScanBlocks = 256;
constexpr uint64_t kScanReady = 1ull << 32;  // flag of a published range sum
constexpr int kScanPer = 8;                   // consecutive vertices per thread in a scan tile

// Empty hash tables (every key empty, reference counts 0), and zero device
// counters and scan status words for the builds that follow; several
// tables in one launch: blockIdx.y picks one.
struct ClearJobs {
  ClearJob job[kMaxLevels];
};

__global__ void __launch_bounds__(kBlock)
k_clear_tables(ClearJobs jobs) {
  const ClearJob& J = jobs.job[blockIdx.y];
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  for (int64_t e = i; e < J.cap; e += stride)
    *reinterpret_cast<uint4*>(&J.entries[e]) = make_uint4(0xffffffffu, 0xffffffffu, 0u, 0u);
  if (i == 0) *static_cast<uint4*>(J.dev_counters) = make_uint4(0u, 0u, 0u, 0u);
  if (i < kScanBlocks) static_cast<uint64_t*>(J.scan_work)[i] = 0ull;
}

// Exclusive prefix sum over the workgroup (wave shuffles, then the four
// wave totals through LDS); *total receives the workgroup sum.
__device__ inline int32_t block_exclusive_sum(int32_t v, int32_t* lds4, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) lds4[wave] = x;
  __syncthreads();
  int32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) {
    const int32_t sw = lds4[w];
    if (w < wave) before += sw;
    tot += sw;
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

// One thread per point.  Embedding: y = E (g/sigma) with E's columns
// orthonormal and orthogonal to 1 (the lattice lives on H_d, coordinates
// summing to zero), scaled by (d+1) sqrt(2/3); a_j folds 1/sigma_j and the
// column norm into one factor.  Coarse levels take the parent's elevated
// position times y_scale (1/2).
// Enclosing simplex (the rounding construction of Adams, Baek and Davis
// 2010, which the paper cites for finding the simplex): round each
// coordinate to the nearest multiple of d+1 (ties down), rank the
// differentials (largest first, equal ones by lower index), move the most
// extreme ones by d+1 until the point lies on H_d, then vertex k adds k to
// every coordinate and subtracts d+1 from the k highest-ranked ones; the
// barycentric weights are the gaps between consecutive sorted differentials.
//
// Outputs per point: slot of each vertex in the global table, its rank in
// that vertex's point list, the weights and the elevated position.  Per new
// vertex: vals[slot] = vertex number, vkeys / vslot by vertex number.
// The slot's count ends as the number of references of the vertex.
// Several levels of one cloud go in one launch, blockIdx.y picking the
// level: a level elevated from the positions and halved l times holds the
// same floats as one halved from its parent's stored elevated positions, so
// no level waits for another.
struct InsertJobs {
  InsertJob job[kMaxLevels];
};

__global__ void __launch_bounds__(kBlock)
k_insert_points(InsertJobs jobs, int64_t m) {
  const InsertJob& J = jobs.job[blockIdx.y];
  const HashView h = J.h;
  uint32_t* const err = J.err;
  __shared__ uint64_t lkey[kLdsSlots];
  __shared__ int32_t lcount[kLdsSlots];
  __shared__ int32_t lslot[kLdsSlots];
  __shared__ int32_t lbase[kLdsSlots];
  __shared__ int32_t ulist[kBlock * kVerts];
  __shared__ int32_t scan_buf[kBlock / 64];
  __shared__ int32_t id_base;

  const int tid = threadIdx.x;
  for (int j = 0; j < kLdsPerThread; ++j) {
    lkey[tid + j * kBlock] = kEmptyKey;
    lcount[tid + j * kBlock] = 0;
  }
  __syncthreads();

  const int64_t p = static_cast<int64_t>(blockIdx.x) * kBlock + tid;
  bool live = p < m;
  bool raised = false;  // this thread set an error bit
  float y[kVerts] = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    if (J.pos != nullptr) {
      const float* __restrict__ pos = J.pos;
      const float g0 = pos[3 * p + 0], g1 = pos[3 * p + 1], g2 = pos[3 * p + 2];
      if (!isfinite(g0) || !isfinite(g1) || !isfinite(g2)) {
        atomicOr(err, kErrNonFinite);
        raised = true;
        live = false;
      } else {
        const float t0 = g0 * J.a0, t1 = g1 * J.a1, t2 = g2 * J.a2;
        float run = 0.0f;
        const float m3 = 3.0f * t2;
        y[3] = run - m3;
        run = run + t2;
        const float m2 = 2.0f * t1;
        y[2] = run - m2;
        run = run + t1;
        const float m1 = 1.0f * t0;
        y[1] = run - m1;
        run = run + t0;
        y[0] = run;
        for (int l = 0; l < J.halvings; ++l)
#pragma unroll
          for (int i = 0; i < kVerts; ++i) y[i] = y[i] * 0.5f;
      }
    } else {
      const float4 v = reinterpret_cast<const float4*>(J.y_in)[p];
      y[0] = v.x * J.y_scale;
      y[1] = v.y * J.y_scale;
      y[2] = v.z * J.y_scale;
      y[3] = v.w * J.y_scale;
    }
    if (J.y_out) reinterpret_cast<float4*>(J.y_out)[p] = make_float4(y[0], y[1], y[2], y[3]);
  }
  if (live) {
    bool ok = true;
    for (int i = 0; i < kVerts; ++i)
      if (!(fabsf(y[i]) < 2.0f * static_cast<float>(kCoordLimit))) ok = false;
    if (!ok) {
      atomicOr(err, isfinite(y[0] + y[1] + y[2] + y[3]) ? kErrKeyRange : kErrNonFinite);
      raised = true;
      live = false;
    }
  }

  float b[kVerts] = {0.f, 0.f, 0.f, 0.f};
  uint64_t keys[kVerts] = {kEmptyKey, kEmptyKey, kEmptyKey, kEmptyKey};
  if (live) {
    int32_t base[kVerts];
    int32_t total = 0;
#pragma unroll
    for (int i = 0; i < kVerts; ++i) {
      const float q = y[i] * 0.25f;
      const float lo = floorf(q) * 4.0f;
      const float hi = lo + 4.0f;
      const float up = hi - y[i];
      const float down = y[i] - lo;
      base[i] = static_cast<int32_t>(up < down ? hi : lo);
      total += base[i];
    }
    const int32_t excess = total / kVerts;
    float diff[kVerts];
#pragma unroll
    for (int i = 0; i < kVerts; ++i) diff[i] = y[i] - static_cast<float>(base[i]);
    int32_t rank[kVerts];
#pragma unroll
    for (int i = 0; i < kVerts; ++i) {
      int32_t r = 0;
#pragma unroll
      for (int j = 0; j < kVerts; ++j)
        r += (diff[j] > diff[i] || (diff[j] == diff[i] && j < i)) ? 1 : 0;
      rank[i] = r;
    }
#pragma unroll
    for (int i = 0; i < kVerts; ++i) {
      if (excess > 0) {
        if (rank[i] >= kVerts - excess) { base[i] -= kVerts; rank[i] += excess - kVerts; }
        else rank[i] += excess;
      } else if (excess < 0) {
        if (rank[i] < -excess) { base[i] += kVerts; rank[i] += kVerts + excess; }
        else rank[i] += excess;
      }
    }
    float z[kVerts];
#pragma unroll
    for (int i = 0; i < kVerts; ++i) {
      const float dz = (y[i] - static_cast<float>(base[i])) * 0.25f;
#pragma unroll
      for (int r = 0; r < kVerts; ++r)
        if (rank[i] == r) z[r] = dz;
    }
    b[0] = 1.0f - (z[0] - z[3]);
    b[1] = z[2] - z[3];
    b[2] = z[1] - z[2];
    b[3] = z[0] - z[1];
#pragma unroll
    for (int k = 0; k < kVerts; ++k) {
      int32_t c[kVerts];
#pragma unroll
      for (int i = 0; i < kVerts; ++i) c[i] = base[i] + k - (rank[i] > kDim - k ? kVerts : 0);
      if (coords_in_range(c[0], c[1], c[2], c[3])) keys[k] = pack_key(c[0], c[1], c[2]);
      else {
        atomicOr(err, kErrKeyRange);
        raised = true;
      }
    }
  }

  // 1. merge the workgroup's references in LDS
  int32_t lsl[kVerts], lrank[kVerts];
#pragma unroll
  for (int k = 0; k < kVerts; ++k) {
    lsl[k] = -1;
    lrank[k] = 0;
    if (keys[k] == kEmptyKey) continue;
    uint32_t s = static_cast<uint32_t>(hash_key(keys[k])) & (kLdsSlots - 1);
    for (int probe = 0; probe < kLdsSlots; ++probe) {
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long*>(&lkey[s]),
                                      static_cast<unsigned long long>(kEmptyKey),
                                      static_cast<unsigned long long>(keys[k]));
      if (prev == kEmptyKey || prev == keys[k]) break;
      s = (s + 1) & (kLdsSlots - 1);
    }
    lsl[k] = static_cast<int32_t>(s);
    lrank[k] = atomicAdd(&lcount[s], 1);
  }
  __syncthreads();

  // 2. compact the distinct keys, then one global insert and one count
  //    update per distinct key, spread over all threads
  int32_t occupied = 0;
  for (int j = 0; j < kLdsPerThread; ++j) occupied += lkey[tid + j * kBlock] != kEmptyKey ? 1 : 0;
  int32_t nunique = 0;
  int32_t at = block_exclusive_sum(occupied, scan_buf, &nunique);
  for (int j = 0; j < kLdsPerThread; ++j) {
    const int sl = tid + j * kBlock;
    if (lkey[sl] != kEmptyKey) ulist[at++] = sl;
  }
  __syncthreads();
  // a thread's distinct keys: u = tid + j * kBlock, j < kVerts (nunique is
  // at most kBlock * kVerts)
  int32_t usl[kVerts], gsl[kVerts];
  uint64_t ukey[kVerts], probe_at[kVerts];
  uint32_t pending = 0;
#pragma unroll
  for (int j = 0; j < kVerts; ++j) {
    const int u = tid + j * kBlock;
    usl[j] = u < nunique ? ulist[u] : 0;
    ukey[j] = lkey[usl[j]];
    probe_at[j] = hash_key(ukey[j]) & h.mask;
    gsl[j] = -1;
    if (u < nunique) pending |= 1u << j;
  }
  uint32_t created_mask = 0;
  for (uint64_t probe = 0; pending != 0 && probe <= h.mask; ++probe) {
    uint64_t prev[kVerts];
#pragma unroll
    for (int j = 0; j < kVerts; ++j)
      if (pending & (1u << j))
        prev[j] = atomicCAS(reinterpret_cast<unsigned long long*>(&h.e[probe_at[j]].key),
                            static_cast<unsigned long long>(kEmptyKey), static_cast<unsigned long long>(ukey[j]));
#pragma unroll
    for (int j = 0; j < kVerts; ++j) {
      if (!(pending & (1u << j))) continue;
      if (prev[j] == kEmptyKey || prev[j] == ukey[j]) {
        gsl[j] = static_cast<int32_t>(probe_at[j]);
        if (prev[j] == kEmptyKey) created_mask |= 1u << j;
        pending &= ~(1u << j);
      } else {
        probe_at[j] = (probe_at[j] + 1) & h.mask;
      }
    }
  }
  if (pending) {
    atomicOr(err, kErrHashFull);
    raised = true;
  }
  // an error bit must have landed before this workgroup counts as finished
  if (raised) __threadfence();
  // reference counts: the returned bases are first needed after the
  // numbering below, so these atomics overlap it
  int32_t gbase[kVerts];
#pragma unroll
  for (int j = 0; j < kVerts; ++j)
    gbase[j] = gsl[j] >= 0 ? atomicAdd(&h.e[gsl[j]].count, lcount[usl[j]]) : 0;
  const int32_t ncreated = __builtin_popcount(created_mask);
  int32_t nblock = 0;
  const int32_t my_first = block_exclusive_sum(ncreated, scan_buf, &nblock);
  // One 64-bit atomic per workgroup claims the numbers of its new vertices
  // (low word: the vertex count) and counts the workgroup as finished with
  // its inserts (high word); the last one copies the count and the error
  // bits into pinned host memory (read by the host after an event).  Error
  // bits are set with atomics, and fenced, before this point in every
  // workgroup.
  if (tid == 0) {
    const unsigned long long old =
        __hip_atomic_fetch_add(reinterpret_cast<unsigned long long*>(J.counter),
                               (1ull << 32) | static_cast<uint32_t>(nblock), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    id_base = static_cast<int32_t>(old & 0xffffffffull);
    if ((old >> 32) == gridDim.x - 1) {
      int32_t* const host_counts = J.host_counts;
      host_counts[0] = id_base + nblock;
      host_counts[1] = static_cast<int32_t>(__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      __threadfence_system();
      host_counts[2] = static_cast<int32_t>(J.stamp);  // the build this readback belongs to
      __threadfence_system();
    }
  }
  __syncthreads();
  int32_t id = id_base + my_first;
#pragma unroll
  for (int j = 0; j < kVerts; ++j) {
    if (tid + j * kBlock < nunique) {
      lslot[usl[j]] = gsl[j];
      lbase[usl[j]] = gbase[j];
    }
    if (!(created_mask & (1u << j))) continue;
    h.e[gsl[j]].val = id;
    J.vkeys[id] = ukey[j];
    J.vslot[id] = gsl[j];
    ++id;
  }
  __syncthreads();

  // 3. per reference: global slot and rank in the vertex's point list
  if (p < m) {
    int32_t so[kVerts], ro[kVerts];
#pragma unroll
    for (int k = 0; k < kVerts; ++k) {
      so[k] = lsl[k] >= 0 ? lslot[lsl[k]] : -1;
      ro[k] = lsl[k] >= 0 ? lbase[lsl[k]] + lrank[k] : 0;
    }
    reinterpret_cast<int4*>(J.slot_out)[p] = make_int4(so[0], so[1], so[2], so[3]);
    reinterpret_cast<int4*>(J.rank_out)[p] = make_int4(ro[0], ro[1], ro[2], ro[3]);
    reinterpret_cast<float4*>(J.w_out)[p] = make_float4(b[0], b[1], b[2], b[3]);
  }

}

__global__ void __launch_bounds__(kBlock)
k_scan(const HashEntry* __restrict__ table, const int32_t* __restrict__ vslot, const int32_t* __restrict__ n_dev,
       uint64_t* __restrict__ status, int32_t* __restrict__ offsets) {
  static_assert(kScanBlocks <= kBlock, "one earlier range per thread");
  __shared__ int32_t lds4[kBlock / 64];
  const int64_t n = *n_dev;
  const int64_t per = (n + kScanBlocks - 1) / kScanBlocks;
  const int64_t beg = blockIdx.x * per, end = min(beg + per, n);
  int32_t s = 0;
  for (int64_t i = beg + threadIdx.x; i < end; i += kBlock) s += table[vslot[i]].count;
  int32_t agg;
  block_exclusive_sum(s, lds4, &agg);
  // the status word carries the sum itself, so relaxed atomics suffice
  if (threadIdx.x == 0)
    __hip_atomic_store(&status[blockIdx.x], kScanReady | static_cast<uint32_t>(agg), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  // thread j < blockIdx.x takes the sum of range j: published, or, should it
  // not appear within a bounded wait, summed here from the counts themselves
  int32_t before = 0;
  const int j = threadIdx.x;
  if (j < static_cast<int>(blockIdx.x)) {
    uint64_t st = 0;
    for (int spin = 0; spin < 100000; ++spin) {
      st = __hip_atomic_load(&status[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (st & kScanReady) break;
      __builtin_amdgcn_s_sleep(2);
    }
    if (st & kScanReady) {
      before = static_cast<int32_t>(static_cast<uint32_t>(st));
    } else {
      const int64_t b2 = j * per, e2 = min(b2 + per, n);
      for (int64_t i = b2; i < e2; ++i) before += table[vslot[i]].count;
    }
  }
  int32_t carry;
  block_exclusive_sum(before, lds4, &carry);  // carry = sum of all earlier ranges
  for (int64_t t0 = beg; t0 < end; t0 += kBlock * kScanPer) {
    const int64_t base = t0 + threadIdx.x * kScanPer;
    int32_t v[kScanPer];
    int32_t loc = 0;
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      v[q] = base + q < end ? table[vslot[base + q]].count : 0;
      loc += v[q];
    }
    int32_t tile_total;
    int32_t run = carry + block_exclusive_sum(loc, lds4, &tile_total);
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      if (base + q < end) offsets[base + q] = run;
      run += v[q];
    }
    carry += tile_total;
  }
  if (end == n && beg < end && threadIdx.x == 0) offsets[n] = carry;
  if (n == 0 && blockIdx.x == 0 && threadIdx.x == 0) offsets[0] = 0;
}

// Per reference e = p*(d+1)+k: vertex index, and its place in J_v:
// entries[offsets[v] + rank] = e with the weight alongside.  The vertex that
// owns list position c*E (E = chunk) is recorded for the chunked splat.
__global__ void __launch_bounds__(kBlock)
k_fill_lists(HashView h, const int32_t* __restrict__ slot, const int32_t* __restrict__ rank,
             const float* __restrict__ w, const int32_t* __restrict__ offsets,
             int32_t* __restrict__ idx, int32_t* __restrict__ entries, float* __restrict__ entry_w,
             int32_t* __restrict__ chunk_first, int chunk, int64_t m4) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (e >= m4) return;
  const int32_t s = slot[e];
  if (s < 0) {
    idx[e] = -1;
    return;
  }
  const int32_t v = h.e[s].val;
  idx[e] = v;
  const int32_t at = offsets[v] + rank[e];
  entries[at] = static_cast<int32_t>(e);
  entry_w[at] = w[e];
  if (at % chunk == 0) chunk_first[at / chunk] = v;
}

// nbr[t][v] for taps 1..8 (tap 0 = v): the vertex at c_v + o_t.
// Entries of the convolution tables (tap t of the vertex with packed key
// `key`; -1 where the target vertex does not exist):
//   same level: the vertex at c_v + o_t (tap 0: the vertex itself);
//   Downsample (coarse vertex into the fine level): the vertex at 2 c_v + o_t;
//   Upsample (fine vertex into the coarse level): the vertex at
//   (c_v + o_t)/2 when that is a lattice point, i.e. even coordinates whose
//   halves agree mod d+1.  The check matters: packed keys omit the last
//   coordinate, so a non-lattice point could otherwise alias a stored key.
__device__ inline int32_t same_level_entry(const HashView& h, uint64_t key, int t) {
  int32_t c[kVerts];
  unpack_key(key, c);
  for (int j = 0; j < kVerts; ++j) c[j] += tap_offset(t, j);
  const uint64_t k = key_or_empty(c);
  return k == kEmptyKey ? -1 : hash_find(h, k);
}

__device__ inline int32_t down_entry(const HashView& fine, uint64_t key, int t) {
  int32_t c[kVerts];
  unpack_key(key, c);
  for (int j = 0; j < kVerts; ++j) c[j] = 2 * c[j] + tap_offset(t, j);
  const uint64_t k = key_or_empty(c);
  return k == kEmptyKey ? -1 : hash_find(fine, k);
}

__device__ inline int32_t up_entry(const HashView& coarse, uint64_t key, int t) {
  int32_t c[kVerts];
  unpack_key(key, c);
  bool lattice_point = true;
  for (int j = 0; j < kVerts; ++j) {
    const int32_t u = c[j] + tap_offset(t, j);
    if (u & 1) lattice_point = false;
    c[j] = u / 2;
  }
  for (int j = 1; j < kVerts; ++j)
    if ((c[j] & 3) != (c[0] & 3)) lattice_point = false;
  if (!lattice_point) return -1;
  const uint64_t k = key_or_empty(c);
  return k == kEmptyKey ? -1 : hash_find(coarse, k);
}

// Convolution tables of one or several levels (blockIdx.y picks the level),
// tap-major (table[t * ld + v]): the same-level table (9 entries per vertex),
// and for a coarse level its Downsample table (9 per coarse vertex) and the
// Upsample table from it into the finer level (9 per fine vertex).  Vertex
// counts come from device memory.
struct TableJobs {
  TableJob job[kMaxLevels];
};

__global__ void __launch_bounds__(kBlock)
k_level_tables(TableJobs jobs) {
  const TableJob& J = jobs.job[blockIdx.y];
  const int64_t nc = *J.n_dev;
  const int64_t nf = J.up ? *J.nf_dev : 0;
  const int64_t per_c = nc * kTaps;
  const int64_t total = J.up ? 2 * per_c + nf * kTaps : per_c;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    if (i < per_c) {
      const int t = static_cast<int>(i / nc);
      const int64_t v = i - static_cast<int64_t>(t) * nc;
      J.nbr[static_cast<int64_t>(t) * J.ld + v] =
          t == 0 ? static_cast<int32_t>(v) : same_level_entry(J.h, J.keys[v], t);
    } else if (i < 2 * per_c) {
      const int64_t k = i - per_c;
      const int t = static_cast<int>(k / nc);
      const int64_t v = k - static_cast<int64_t>(t) * nc;
      J.down[static_cast<int64_t>(t) * J.ld + v] = down_entry(J.hf, J.keys[v], t);
    } else {
      const int64_t k = i - 2 * per_c;
      const int t = static_cast<int>(k / nf);
      const int64_t v = k - static_cast<int64_t>(t) * nf;
      J.up[static_cast<int64_t>(t) * J.ldf + v] = up_entry(J.h, J.fkeys[v], t);
    }
  }
}

// Row order for a convolution table: within each range of kOrderRange rows,
// rows are grouped by their tap mask (bit t set when tap t is present) with
// a counting sort in LDS.  Tiles of the convolution then mostly hold rows of
// one mask and skip the taps none of their rows uses, while the order stays
// local, so the gather keeps its spatial locality.  The order within a mask
// depends on scheduling; the convolution's result for a row does not.
constexpr int kOrderRange = 4096;

constexpr int kOrderThreads = 1024;

// Several tables ordered in one launch: blockIdx.y picks the table.
struct MaskOrderJobs {
  RowOrderJob job[kMaxRowOrderJobs];
};

__global__ void __launch_bounds__(kOrderThreads)
k_mask_order(MaskOrderJobs jobs) {
  const RowOrderJob& J = jobs.job[blockIdx.y];
  const int32_t* __restrict__ nbr = J.nbr;
  const int64_t ldn = J.ld;
  const int32_t* __restrict__ n_dev = J.n_dev;
  int32_t* __restrict__ rows = J.rows;
  __shared__ int32_t hist[kMaskBins];
  __shared__ int32_t wave_sum[kMaskBins / 64];
  __shared__ uint16_t mk[kOrderRange];
  __shared__ uint16_t rk[kOrderRange];
  constexpr int kPer = kOrderRange / kOrderThreads;  // rows per thread, loaded together
  static_assert(kMaskBins <= kOrderThreads, "one bin per thread");
  const int tid = threadIdx.x;
  const int64_t n = *n_dev;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kOrderRange;
  if (r0 >= n) return;
  const int cnt = static_cast<int>(n - r0 < kOrderRange ? n - r0 : kOrderRange);
  if (tid < kMaskBins) hist[tid] = 0;
  __syncthreads();
  int m[kPer];
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = b * kOrderThreads + tid;
    m[b] = 0;
    if (i < cnt) {
#pragma unroll
      for (int t = 0; t < kTaps; ++t)
        if (nbr[static_cast<int64_t>(t) * ldn + r0 + i] >= 0) m[b] |= 1 << t;
    }
  }
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = b * kOrderThreads + tid;
    if (i < cnt) {
      mk[i] = static_cast<uint16_t>(m[b]);
      rk[i] = static_cast<uint16_t>(atomicAdd(&hist[m[b]], 1));
    }
  }
  __syncthreads();
  // exclusive scan of the 512 bins, one per thread of the first 512
  const int lane = tid & 63, wave = tid >> 6;
  int32_t x = tid < kMaskBins ? hist[tid] : 0;
  const int32_t own = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (tid < kMaskBins && lane == 63) wave_sum[wave] = x;
  __syncthreads();
  int32_t before = 0;
  for (int w = 0; w < wave && w < kMaskBins / 64; ++w) before += wave_sum[w];
  __syncthreads();
  if (tid < kMaskBins) hist[tid] = before + x - own;  // now the start of each mask
  __syncthreads();
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = b * kOrderThreads + tid;
    if (i < cnt) rows[r0 + hist[mk[i]] + rk[i]] = static_cast<int32_t>(r0 + i);
  }
}

__global__ void __launch_bounds__(kBlock)
k_export_keys(const uint64_t* __restrict__ vkeys, int64_t n, int4* __restrict__ out) {
  const int64_t v = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (v >= n) return;
  int32_t c[kVerts];
  unpack_key(vkeys[v], c);
  out[v] = make_int4(c[0], c[1], c[2], c[3]);
}

__global__ void __launch_bounds__(kBlock)
k_transpose_table(const int32_t* __restrict__ tab, int64_t ld, int64_t n, int32_t* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n * kTaps) return;
  const int64_t v = i / kTaps;
  const int t = static_cast<int>(i - v * kTaps);
  out[i] = tab[static_cast<int64_t>(t) * ld + v];
}

// Number of entries >= 0 among the first n rows of a tap-major table: the
// (row, tap) pairs whose neighbour exists.  Integer sums, so the count does
// not depend on the order of the atomics.
__global__ void __launch_bounds__(kBlock)
k_count_taps(const int32_t* __restrict__ tab, int64_t ld, int64_t n, unsigned long long* __restrict__ count) {
  __shared__ unsigned long long part[kBlock / 64];
  unsigned long long c = 0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n * kTaps;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t t = i / n, v = i - t * n;
    c += tab[t * ld + v] >= 0 ? 1u : 0u;
  }
  for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long s = 0;
    for (int w = 0; w < kBlock / 64; ++w) s += part[w];
    atomicAdd(count, s);
  }
}

inline unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kBlock - 1) / kBlock); }

}  // namespace

void launch_clear_table(HashEntry* keys, int64_t cap, void* dev_counters, void* scan_work, hipStream_t s) {
  const ClearJob job{keys, cap, dev_counters, scan_work};
  launch_clear_tables(&job, 1, s);
}

void launch_insert_levels(const InsertJob* jobs, const hipEvent_t* done, int n, int64_t m, hipStream_t s) {
  if (n <= 0) return;
  if (m > 0) {
    InsertJobs all{};
    for (int i = 0; i < n; ++i) all.job[i] = jobs[i];
    ScopedKernelTimer tm("insert", s);
    launch_signal(k_insert_points, dim3(blocks_for(m), n), dim3(kBlock), 0, s, done[0], all, m);
  } else {
    (void)hipEventRecord(done[0], s);
  }
  for (int i = 1; i < n; ++i) (void)hipEventRecord(done[i], s);
}

int64_t scan_workspace_bytes() { return kScanBlocks * sizeof(uint64_t); }

void launch_count_scan(const HashEntry* table, const int32_t* vslot, const int32_t* n_dev,
                       int32_t* offsets, void* work, hipStream_t s) {
  ScopedKernelTimer tm("scan", s);
  launch(k_scan, dim3(kScanBlocks), dim3(kBlock), 0, s, table, vslot, n_dev,
                     static_cast<uint64_t*>(work), offsets);
}

void launch_fill_lists(HashView h, const int32_t* slot, const int32_t* rank, const float* w,
                       const int32_t* offsets, int32_t* idx, int32_t* entries, float* entry_w,
                       int32_t* chunk_first, int chunk, int64_t m4, hipStream_t s) {
  if (m4 <= 0) return;
  ScopedKernelTimer tm("lists", s);
  launch(k_fill_lists, dim3(blocks_for(m4)), dim3(kBlock), 0, s, h, slot, rank, w, offsets,
                     idx, entries, entry_w, chunk_first, chunk, m4);
}

// grid for a grid-stride pass over up to `work` items
inline unsigned stride_grid(int64_t work) {
  const int64_t b = (work + kBlock - 1) / kBlock;
  return static_cast<unsigned>(b < 1 ? 1 : (b < 4096 ? b : 4096));
}

void launch_neighbor_table(HashView h, const uint64_t* vkeys, const int32_t* n_dev, int64_t n_max,
                           int32_t* nbr, int64_t ldn, int32_t* nbr_rows, hipStream_t s, RowOrderBatch* defer) {
  if (n_max <= 0) return;
  TableJob j{};
  j.h = h;
  j.keys = vkeys;
  j.n_dev = n_dev;
  j.nbr = nbr;
  j.ld = ldn;
  launch_level_tables(&j, 1, n_max * kTaps, s);
  RowOrderBatch own;
  RowOrderBatch& b = defer ? *defer : own;
  b.add(RowOrderJob{nbr, ldn, n_dev, nbr_rows}, n_max);
  if (!defer) launch_row_orders(b, nullptr, s);
}

void launch_coarse_tables(HashView coarse, HashView fine, const uint64_t* coarse_keys, const uint64_t* fine_keys,
                          const int32_t* nc_dev, const int32_t* nf_dev, int64_t nc_max, int64_t nf_max, int32_t* nbr,
                          int32_t* down, int32_t* up, int32_t* up_rows, int32_t* nbr_rows, int32_t* down_rows,
                          hipEvent_t done, hipStream_t s, RowOrderBatch* defer) {
  if (nc_max <= 0 || nf_max <= 0) {
    if (done) (void)hipEventRecord(done, s);
    return;
  }
  TableJob j{coarse, fine, coarse_keys, fine_keys, nc_dev, nf_dev, nbr, down, up, nc_max, nf_max};
  launch_level_tables(&j, 1, (2 * nc_max + nf_max) * kTaps, s);
  // the rows of all three tables grouped by tap mask, in one launch (or in
  // the caller's batch)
  RowOrderBatch own;
  RowOrderBatch& b = defer ? *defer : own;
  b.add(RowOrderJob{up, nf_max, nf_dev, up_rows}, nf_max);
  b.add(RowOrderJob{nbr, nc_max, nc_dev, nbr_rows}, nc_max);
  b.add(RowOrderJob{down, nc_max, nc_dev, down_rows}, nc_max);
  if (!defer) launch_row_orders(b, done, s);
}

void launch_level_tables(const TableJob* jobs, int n, int64_t work_max, hipStream_t s) {
  if (n <= 0 || work_max <= 0) return;
  TableJobs all{};
  for (int i = 0; i < n; ++i) all.job[i] = jobs[i];
  ScopedKernelTimer tm("nbr", s);
  launch(k_level_tables, dim3(stride_grid(work_max), static_cast<unsigned>(n)), dim3(kBlock), 0, s, all);
}

void launch_row_orders(const RowOrderBatch& b, hipEvent_t done, hipStream_t s) {
  if (b.n == 0 || b.max_rows <= 0) {
    if (done) (void)hipEventRecord(done, s);
    return;
  }
  ScopedKernelTimer tm("nbr", s);
  MaskOrderJobs jobs{};
  for (int i = 0; i < b.n; ++i) jobs.job[i] = b.job[i];
  const dim3 grid(static_cast<unsigned>((b.max_rows + kOrderRange - 1) / kOrderRange), static_cast<unsigned>(b.n));
  if (done)
    launch_signal(k_mask_order, grid, dim3(kOrderThreads), 0, s, done, jobs);
  else
    launch(k_mask_order, grid, dim3(kOrderThreads), 0, s, jobs);
}

void launch_clear_tables(const ClearJob* jobs, int n, hipStream_t s) {
  if (n <= 0) return;
  ClearJobs J{};
  int64_t cap_max = 0;
  for (int i = 0; i < n; ++i) {
    J.job[i] = jobs[i];
    cap_max = std::max(cap_max, jobs[i].cap);
  }
  const int64_t want = (cap_max + kBlock * 4 - 1) / (kBlock * 4);
  const unsigned grid = static_cast<unsigned>(want < 1 ? 1 : (want < 8192 ? want : 8192));
  ScopedKernelTimer tm("fill", s);
  launch(k_clear_tables, dim3(grid, static_cast<unsigned>(n)), dim3(kBlock), 0, s, J);
}

void launch_export_keys(const uint64_t* vkeys, int64_t n, int32_t* out, hipStream_t s) {
  if (n <= 0) return;
  launch(k_export_keys, dim3(blocks_for(n)), dim3(kBlock), 0, s, vkeys, n,
                     reinterpret_cast<int4*>(out));
}

void launch_count_taps(const int32_t* tab, int64_t ld, int64_t n, unsigned long long* count, hipStream_t s) {
  if (n <= 0) return;
  launch(k_count_taps, dim3(static_cast<unsigned>(std::min<int64_t>((n * kTaps + kBlock - 1) / kBlock, 1024))),
         dim3(kBlock), 0, s, tab, ld, n, count);
}

void launch_transpose_table(const int32_t* tab, int64_t ld, int64_t n, int32_t* out, hipStream_t s) {
  if (n <= 0) return;
  launch(k_transpose_table, dim3(blocks_for(n * kTaps)), dim3(kBlock), 0, s, tab, ld, n, out);
}

}  // namespace lat

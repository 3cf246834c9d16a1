// liblattice C ABI: argument validation, handle lifetime, device memory and
// kernel-family timing.  Every lattice operation is a hand-written kernel in
// create.hip, splat_slice.hip or conv.hip; this file only orchestrates them.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstddef>
#include <cstdio>
#include <cstring>
#include <deque>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "lattice_internal.h"

namespace lat {
int splat_max_channels(bool bf16);
int deform_max_channels(bool bf16);
}

using namespace lat;

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
namespace {

thread_local std::string g_last_error;

int fail(int status, const std::string& msg) {
  g_last_error = std::string(lattice_status_string(status)) + ": " + msg;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(LAT_EDEVICE, std::string(what) + " failed: " + hipGetErrorString(e));
}

#define HIP_TRY(expr)                                  \
  do {                                                 \
    hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return hip_fail(e_, #expr);  \
  } while (0)

// ---------------------------------------------------------------------------
// caching device allocator: freed blocks are kept per (device, size class)
// and handed out again without hipMalloc.  A block goes back first to the
// stream that released it; else to another stream once the releasing stream
// has drained (hipStreamQuery).  While that stream is still busy the pool
// allocates a new block rather than wait, so steps on two streams that take
// turns with the same scratch sizes each end up with blocks of their own and
// run side by side; only when a size class already holds kMaxIdle blocks of
// busy streams does the caller's thread wait for one (hipStreamSynchronize).
// Nothing is recorded at a release: an event per release cost the host
// more than the rest of a training step's scratch handling.
// ---------------------------------------------------------------------------
struct Block {
  void* ptr;
  size_t bytes;
  hipStream_t stream;
};

class Pool {
 public:
  static constexpr size_t kMaxIdle = 4;   // idle blocks of busy streams per size class before waiting

  static Pool& get() {
    static Pool* p = new Pool();   // never destroyed: blocks live until exit
    return *p;
  }

  static size_t size_class(size_t bytes) {
    size_t c = 256;
    while (c < bytes) c <<= 1;
    return c;
  }

  int alloc(size_t bytes, hipStream_t s, void** out) {
    *out = nullptr;
    if (bytes == 0) return LAT_OK;
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    const size_t cls = size_class(bytes);
    {
      std::lock_guard<std::mutex> lk(mu_);
      auto& lst = free_[{dev, cls}];
      for (size_t i = 0; i < lst.size(); ++i) {
        if (lst[i].stream == s) {
          *out = lst[i].ptr;
          lst.erase(lst.begin() + static_cast<long>(i));
          return LAT_OK;
        }
      }
      for (size_t i = 0; i < lst.size(); ++i) {
        const hipError_t q = hipStreamQuery(lst[i].stream);
        if (q == hipSuccess) {
          *out = lst[i].ptr;
          lst.erase(lst.begin() + static_cast<long>(i));
          return LAT_OK;
        }
        (void)hipGetLastError();   // hipErrorNotReady is not an error of a later call
      }
      if (lst.size() >= kMaxIdle) {
        Block b = lst.back();
        lst.pop_back();
        HIP_TRY(hipStreamSynchronize(b.stream));
        *out = b.ptr;
        return LAT_OK;
      }
    }
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, cls);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      trim(dev);
      e = hipMalloc(&p, cls);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(LAT_ENOMEM, "hipMalloc of " + std::to_string(cls) + " bytes");
      }
    }
    *out = p;
    return LAT_OK;
  }

  void release(void* p, size_t bytes, hipStream_t s) {
    const std::pair<void*, size_t> one{p, bytes};
    release_all(&one, 1, s);
  }

  // Blocks whose last uses are queued on stream s.
  void release_all(const std::pair<void*, size_t>* bufs, size_t n, hipStream_t s) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return;
    std::lock_guard<std::mutex> lk(mu_);
    for (size_t i = 0; i < n; ++i)
      if (bufs[i].first && bufs[i].second != 0)
        free_[{dev, size_class(bufs[i].second)}].push_back(Block{bufs[i].first, bufs[i].second, s});
    ++releases_[s];
  }

  // Number of releases to stream s so far (a block released later may still
  // have uses pending on s).
  uint64_t release_count(hipStream_t s) {
    std::lock_guard<std::mutex> lk(mu_);
    auto it = releases_.find(s);
    return it == releases_.end() ? 0 : it->second;
  }

 private:
  void trim(int dev) {
    std::lock_guard<std::mutex> lk(mu_);
    (void)hipDeviceSynchronize();
    for (auto& kv : free_) {
      if (kv.first.first != dev) continue;
      for (auto& b : kv.second) (void)hipFree(b.ptr);
      kv.second.clear();
    }
  }

  std::mutex mu_;
  std::map<std::pair<int, size_t>, std::vector<Block>> free_;
  std::map<hipStream_t, uint64_t> releases_;
};

// ---------------------------------------------------------------------------
// kernel-family timing with events on the launch stream
// ---------------------------------------------------------------------------
struct TimerFamily {
  std::string name;
  bool enabled = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> recorded;
  std::vector<hipEvent_t> spare;
};

std::mutex g_timer_mu;
std::deque<TimerFamily>& timer_families() {
  static auto* v = new std::deque<TimerFamily>();  // stable element addresses
  return *v;
}
bool g_any_timer = false;

TimerFamily* find_family(const char* name, bool create) {
  auto& fams = timer_families();
  for (auto& f : fams)
    if (f.name == name) return &f;
  if (!create) return nullptr;
  fams.push_back(TimerFamily{});
  fams.back().name = name;
  return &fams.back();
}

hipEvent_t take_event(TimerFamily* f) {
  if (!f->spare.empty()) {
    hipEvent_t e = f->spare.back();
    f->spare.pop_back();
    return e;
  }
  // timing events: no system-scope fence when they complete (only device
  // timestamps are read from them)
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

namespace lat {

thread_local TimerFamily* t_active = nullptr;  // family of the live ScopedKernelTimer

thread_local int t_depth = 0;  // nesting of live ScopedKernelTimers; the outermost names the family

void timer_begin(const char* family) {
  if (t_depth++ > 0) return;
  t_active = nullptr;
  if (!g_any_timer) return;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  TimerFamily* f = find_family(family, false);
  if (f && f->enabled) t_active = f;
}

void timer_end() {
  if (--t_depth == 0) t_active = nullptr;
}

bool timer_take_events(hipEvent_t* start, hipEvent_t* stop) {
  if (!t_active) return false;
  std::lock_guard<std::mutex> lk(g_timer_mu);
  hipEvent_t a = take_event(t_active), b = a ? take_event(t_active) : nullptr;
  if (!a || !b) {
    if (a) t_active->spare.push_back(a);
    return false;
  }
  t_active->recorded.emplace_back(a, b);
  *start = a;
  *stop = b;
  return true;
}

}  // namespace lat

// ---------------------------------------------------------------------------
// handle
// ---------------------------------------------------------------------------
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

struct DeviceCounters {
  int32_t counter;  // vertex count; with `done`, one 64-bit word updated atomically
  uint32_t done;    // workgroups of the insert kernel past their vertex claims
  uint32_t err;     // error bits
  uint32_t pad;
};
static_assert(offsetof(DeviceCounters, done) == 4, "count and done share one aligned 64-bit word");

// Pinned host landing slot, written by the last workgroup of the insert
// kernel: [0] vertex count, [1] error bits, then [2] the stamp of the build.
struct HostCounts {
  int32_t n;
  uint32_t err;
  uint32_t stamp;
  uint32_t pad;
};

struct lattice_s {
  int level = 0;
  double scale[3] = {1.0, 1.0, 1.0};  // sigma_j * 2^level: positions in lattice units are pos / scale
  int64_t m = 0;
  int64_t n = 0;                 // valid once counts_known
  int64_t nmax = 0;              // host-side bound on n (buffer sizes)
  int64_t cap = 0;               // hash slots
  bool counts_known = true;      // n and the device error flag have been read back
  DeviceCounters* dc = nullptr;  // device counters (vertex count, error bits)
  HostCounts* host_dc = nullptr;  // pinned landing slot of their readback
  hipEvent_t counts_ready = nullptr;  // recorded after the readback
  int32_t* host_counts_dev = nullptr;  // device view of host_dc (the insert's landing slot)
  int chunk = 64;                // list entries per splat work item
  int status = LAT_OK;           // poisoned when != LAT_OK
  int children = 0;
  lattice_s* parent = nullptr;
  hipStream_t stream = nullptr;  // the caller's stream: owner of the handle's buffers
  hipStream_t bstream = nullptr;  // stream the build ran on (the library's side stream for a coarse level)
  uint64_t side_seq = 0;          // built on the side stream: its build's number there (0: not)
  hipEvent_t built = nullptr;     // side-stream build: completes with its last kernel
  hipEvent_t rebuilt = nullptr;   // after a rebuild (overflow, or a rebuilt parent) on the owner stream
  std::vector<hipStream_t> rebuilt_joined;  // other streams already ordered after it
  std::vector<hipStream_t> joined;  // streams already ordered after that build
  uint64_t releases_at_insert = 0;  // owner pool's release count when the insert was enqueued
  std::vector<DevBuf> owned;

  float* y = nullptr;            // m x 4 elevated positions
  int32_t* idx = nullptr;        // m x 4 simplex vertex indices
  float* w = nullptr;            // m x 4 barycentric weights
  HashEntry* table = nullptr;    // hash table (cap entries of key + vertex number)
  uint64_t* vkeys = nullptr;     // n packed vertex keys
  int32_t* offsets = nullptr;    // n+1 list offsets of J_v
  int32_t* entries = nullptr;    // 4m entries p*4+k grouped by vertex
  float* entry_w = nullptr;      // 4m weights of those entries
  int32_t* chunk_first = nullptr;  // vertex owning list position c * kSplatChunk
  int64_t total = 0;               // number of list entries (4m)
  int32_t* nbr = nullptr;        // 9 x nmax same-level table (tap-major, ld nmax)
  int32_t* down = nullptr;       // 9 x nmax table into the parent (coarse levels, ld nmax)
  int32_t* up = nullptr;         // 9 x parent->nmax table from the parent into this level
  int32_t* up_rows = nullptr;    // parent vertices, grouped by the tap mask of their up row
  int32_t* nbr_rows = nullptr;   // this level's vertices grouped by the tap mask of their same-level row
  int32_t* down_rows = nullptr;  // this level's vertices grouped by the tap mask of their down row
  int64_t retry_cap = 0;          // coarse levels: table size of a rebuild after overflow
  uint32_t stamp = 0;             // stamp of the current build's count readback
  uint64_t generation = 0;        // rebuilds of this handle after an overflow
  uint64_t parent_generation = 0; // the parent's generation this level was built from
  // A coarse level builds its vertex lists J_v (and the per-point vertex
  // indices) only when an operator first needs them: the convolutions only
  // need the tables.  Until then it keeps what the list build reads.
  bool lists_ready = true;
  bool defer_lists = false;       // a coarse level: lists built on first use
  int32_t* vslot = nullptr;       // per vertex: its slot
  int32_t* slot = nullptr;        // per reference: slot of its vertex
  int32_t* rank = nullptr;        // per reference: rank within its vertex
  void* scan_work = nullptr;      // status words of the count scan (cleared by the build)

  HashView hash() const { return HashView{table, static_cast<uint64_t>(cap - 1)}; }

  int alloc(size_t bytes, hipStream_t s, void** out) {
    const int st = Pool::get().alloc(bytes, s, out);
    if (st == LAT_OK && *out) owned.push_back(DevBuf{*out, bytes});
    return st;
  }

  bool joined_by(hipStream_t s) const {
    for (hipStream_t j : joined)
      if (j == s) return true;
    return false;
  }

  // Buffers go back to the pool of the owner stream, which must first be
  // ordered after a side-stream build.
  void free_all();
};

namespace {

// Pinned host slots for the counter readbacks and a pool of events; both are
// recycled when handles are destroyed.
class HostSlots {
 public:
  static HostSlots& get() {
    static HostSlots* h = new HostSlots();
    return *h;
  }
  HostCounts* take() {
    std::lock_guard<std::mutex> lk(mu_);
    if (free_.empty()) {
      void* p = nullptr;
      constexpr int kSlab = 256;
      if (hipHostMalloc(&p, sizeof(HostCounts) * kSlab, hipHostMallocDefault) != hipSuccess) return nullptr;
      for (int i = 0; i < kSlab; ++i) free_.push_back(static_cast<HostCounts*>(p) + i);
    }
    HostCounts* d = free_.back();
    free_.pop_back();
    return d;
  }
  void give(HostCounts* d) {
    if (!d) return;
    std::lock_guard<std::mutex> lk(mu_);
    free_.push_back(d);
  }
  hipEvent_t take_event() {
    std::lock_guard<std::mutex> lk(mu_);
    if (!events_.empty()) {
      hipEvent_t e = events_.back();
      events_.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
    return e;
  }
  void give_event(hipEvent_t e) {
    if (!e) return;
    std::lock_guard<std::mutex> lk(mu_);
    events_.push_back(e);
  }

 private:
  std::mutex mu_;
  std::vector<HostCounts*> free_;
  std::vector<hipEvent_t> events_;
};

int64_t next_pow2(int64_t v) {
  int64_t c = 1;
  while (c < v) c <<= 1;
  return c;
}

int status_from_err_bits(uint32_t bits) {
  if (bits & kErrNonFinite) return LAT_ENONFINITE;
  if (bits & kErrKeyRange) return LAT_EKEYRANGE;
  if (bits & kErrHashFull) return LAT_EHASHFULL;
  return LAT_OK;
}

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, what);
  return LAT_OK;
}

// Scratch buffer from the pool, returned when the scope ends.
struct Scratch {
  void* p = nullptr;
  size_t bytes = 0;
  hipStream_t s = nullptr;
  ~Scratch() { Pool::get().release(p, bytes, s); }
  int get(size_t b, hipStream_t st) {
    bytes = b;
    s = st;
    return Pool::get().alloc(b, st, &p);
  }
  template <class T> T* as() const { return static_cast<T*>(p); }
};

// Enqueue the construction of a lattice with a table of `cap` slots:
// clear, insert (whose last workgroup writes the vertex count and the error
// bits into the pinned host slot; an event marks its completion), then the
// scan, the vertex lists and the tables, which take the vertex count from
// device memory.  Nothing waits here.
// A build in three parts, so that the levels of a hierarchy can share
// launches (lattice_create_hierarchy): prepare_build sizes and allocates
// the level and takes its host slots (no device work), issue_insert
// enqueues the insert (the table must have been cleared on s before),
// issue_tables the lists (finest level) and the neighbour tables, with the
// row orders added to `defer` when given instead of launched.
int prepare_build(lattice_s* L, const lattice_s* parent, int64_t cap, hipStream_t s) {
  const int64_t m = L->m;
  const int64_t refs = 4 * m;
  const int64_t nmax = std::min(cap, refs);
  L->cap = cap;
  L->nmax = nmax;
  L->total = refs;
  L->chunk = refs >= 64 * 32768 ? 64 : (refs >= 32 * 32768 ? 32 : 16);
  const int64_t nchunks = (refs + L->chunk - 1) / L->chunk;
  L->bstream = s;
  int st;
  // One pool block per build, carved into the handle's buffers (256-byte
  // aligned); the elevated positions come first, so the block's address is
  // theirs.
  size_t off = 0;
  auto carve = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) & ~static_cast<size_t>(255);
    return o;
  };
  const size_t o_y = carve(sizeof(float) * 4 * m);
  const size_t o_idx = carve(sizeof(int32_t) * refs);
  const size_t o_w = carve(sizeof(float) * refs);
  const size_t o_table = carve(sizeof(HashEntry) * cap);
  const size_t o_vkeys = carve(sizeof(uint64_t) * nmax);
  const size_t o_dc = carve(sizeof(DeviceCounters));
  const size_t o_offsets = carve(sizeof(int32_t) * (nmax + 1));
  const size_t o_entries = carve(sizeof(int32_t) * refs);
  const size_t o_entry_w = carve(sizeof(float) * refs);
  const size_t o_chunk_first = carve(sizeof(int32_t) * nchunks);
  const size_t o_nbr = carve(sizeof(int32_t) * kTaps * nmax);
  const size_t o_down = parent ? carve(sizeof(int32_t) * kTaps * nmax) : 0;
  const size_t o_up = parent ? carve(sizeof(int32_t) * kTaps * parent->nmax) : 0;
  const size_t o_up_rows = parent ? carve(sizeof(int32_t) * parent->nmax) : 0;
  const size_t o_nbr_rows = carve(sizeof(int32_t) * nmax);
  const size_t o_down_rows = parent ? carve(sizeof(int32_t) * nmax) : 0;
  // The finest level builds its lists now (splat needs them); a coarse level
  // when an operator first needs them.  Either way the inputs of the list
  // build are the handle's own buffers: a build releases nothing to the
  // pool, so a coarse level can start after the finer level's insert.
  const bool defer_lists = parent != nullptr;
  const size_t o_vslot = carve(sizeof(int32_t) * nmax);
  const size_t o_slot = carve(sizeof(int32_t) * refs);
  const size_t o_rank = carve(sizeof(int32_t) * refs);
  const size_t o_work = carve(static_cast<size_t>(scan_workspace_bytes()));
  void* blk = nullptr;
  if ((st = L->alloc(off, L->stream, &blk)) != LAT_OK) return st;
  auto at = [&](size_t o) { return static_cast<void*>(static_cast<char*>(blk) + o); };
  L->y = static_cast<float*>(at(o_y));
  L->idx = static_cast<int32_t*>(at(o_idx));
  L->w = static_cast<float*>(at(o_w));
  L->table = static_cast<HashEntry*>(at(o_table));
  L->vkeys = static_cast<uint64_t*>(at(o_vkeys));
  L->dc = static_cast<DeviceCounters*>(at(o_dc));
  L->offsets = static_cast<int32_t*>(at(o_offsets));
  L->entries = static_cast<int32_t*>(at(o_entries));
  L->entry_w = static_cast<float*>(at(o_entry_w));
  L->chunk_first = static_cast<int32_t*>(at(o_chunk_first));
  L->nbr = static_cast<int32_t*>(at(o_nbr));
  L->nbr_rows = static_cast<int32_t*>(at(o_nbr_rows));
  if (parent) {
    L->down = static_cast<int32_t*>(at(o_down));
    L->up = static_cast<int32_t*>(at(o_up));
    L->up_rows = static_cast<int32_t*>(at(o_up_rows));
    L->down_rows = static_cast<int32_t*>(at(o_down_rows));
  }
  L->vslot = static_cast<int32_t*>(at(o_vslot));
  L->slot = static_cast<int32_t*>(at(o_slot));
  L->rank = static_cast<int32_t*>(at(o_rank));
  L->scan_work = at(o_work);
  if (!L->host_dc && !(L->host_dc = HostSlots::get().take())) return fail(LAT_ENOMEM, "pinned host slot");
  if (!L->counts_ready && !(L->counts_ready = HostSlots::get().take_event()))
    return fail(LAT_EDEVICE, "event creation failed");

  HIP_TRY(hipHostGetDevicePointer(reinterpret_cast<void**>(&L->host_counts_dev), L->host_dc, 0));
  static std::atomic<uint32_t> g_stamp{0};
  L->stamp = m > 0 ? ++g_stamp : 0;
  L->host_dc->stamp = ~L->stamp;
  L->defer_lists = defer_lists;
  // unknown until the insert reports (a coarser level prepared before this
  // one's insert is enqueued must not size its table from n = 0)
  L->counts_known = false;
  return LAT_OK;
}

// The insert of level L: from the positions (halved `halvings` times after
// elevation) or from y_src times y_scale.
InsertJob insert_job(const lattice_s* L, const float* pos, const float* y_src, float y_scale, int halvings,
                     const float a[3]) {
  InsertJob j{};
  j.pos = pos;
  j.y_in = y_src;
  j.y_scale = y_scale;
  j.halvings = halvings;
  j.a0 = a[0];
  j.a1 = a[1];
  j.a2 = a[2];
  j.h = L->hash();
  j.counter = &L->dc->counter;
  j.vkeys = L->vkeys;
  j.vslot = L->vslot;
  j.slot_out = L->slot;
  j.rank_out = L->rank;
  j.w_out = L->w;
  j.y_out = L->y;
  j.err = &L->dc->err;
  j.host_counts = L->host_counts_dev;
  j.stamp = L->stamp;
  return j;
}

// inserts of n levels of one cloud in one launch (each table cleared on s before)
int issue_inserts(lattice_s* const* Ls, const InsertJob* jobs, int n, hipStream_t s) {
  hipEvent_t done[kMaxLevels];
  for (int i = 0; i < n; ++i) done[i] = Ls[i]->counts_ready;
  launch_insert_levels(jobs, done, n, Ls[0]->m, s);
  for (int i = 0; i < n; ++i) {
    Ls[i]->releases_at_insert = Pool::get().release_count(Ls[i]->stream);
    Ls[i]->counts_known = false;
  }
  HIP_TRY(hipGetLastError());
  return LAT_OK;
}

int issue_insert(lattice_s* L, const float* pos, const float* y_src, float y_scale, const float a[3], hipStream_t s) {
  const InsertJob j = insert_job(L, pos, y_src, y_scale, 0, a);
  return issue_inserts(&L, &j, 1, s);
}

// the point lists J_v, unless the level builds them on first use
void issue_lists(lattice_s* L, hipStream_t s) {
  L->lists_ready = !L->defer_lists;
  if (!L->defer_lists) {
    launch_count_scan(L->table, L->vslot, &L->dc->counter, L->offsets, L->scan_work, s);
    launch_fill_lists(L->hash(), L->slot, L->rank, L->w, L->offsets, L->idx, L->entries, L->entry_w,
                      L->chunk_first, L->chunk, L->total, s);
  }
}

// level L's convolution tables (parent: the finer level, or null)
TableJob table_job(const lattice_s* L, const lattice_s* parent, int64_t* work) {
  TableJob j{};
  j.h = L->hash();
  j.keys = L->vkeys;
  j.n_dev = &L->dc->counter;
  j.nbr = L->nbr;
  j.ld = L->nmax;
  *work = L->nmax * kTaps;
  if (parent) {
    j.hf = parent->hash();
    j.fkeys = parent->vkeys;
    j.nf_dev = &parent->dc->counter;
    j.down = L->down;
    j.up = L->up;
    j.ldf = parent->nmax;
    *work = (2 * L->nmax + parent->nmax) * kTaps;
  }
  return j;
}

// the row orders of level L's tables, added to b (launched first when b is full)
void add_row_orders(RowOrderBatch& b, const lattice_s* L, const lattice_s* parent, hipStream_t s) {
  if (b.n + (parent ? 3 : 1) > kMaxRowOrderJobs) {
    launch_row_orders(b, nullptr, s);
    b = RowOrderBatch{};
  }
  const int32_t* n_dev = &L->dc->counter;
  if (parent) b.add(RowOrderJob{L->up, parent->nmax, &parent->dc->counter, L->up_rows}, parent->nmax);
  b.add(RowOrderJob{L->nbr, L->nmax, n_dev, L->nbr_rows}, L->nmax);
  if (parent) b.add(RowOrderJob{L->down, L->nmax, n_dev, L->down_rows}, L->nmax);
}

void issue_tables(lattice_s* L, const lattice_s* parent, hipEvent_t built, hipStream_t s, RowOrderBatch* defer) {
  const int32_t* n_dev = &L->dc->counter;
  issue_lists(L, s);
  if (parent)
    launch_coarse_tables(L->hash(), parent->hash(), L->vkeys, parent->vkeys, n_dev, &parent->dc->counter, L->nmax,
                         parent->nmax, L->nbr, L->down, L->up, L->up_rows, L->nbr_rows, L->down_rows, built, s,
                         defer);
  else
    launch_neighbor_table(L->hash(), L->vkeys, n_dev, L->nmax, L->nbr, L->nmax, L->nbr_rows, s, defer);
}

int enqueue_build(lattice_s* L, const float* pos, const float* y_src, float y_scale, const float a[3],
                  const lattice_s* parent, int64_t cap, hipStream_t s, hipEvent_t built = nullptr) {
  int st;
  if ((st = prepare_build(L, parent, cap, s)) != LAT_OK) return st;
  launch_clear_table(L->table, cap, L->dc, L->scan_work, s);
  if ((st = issue_insert(L, pos, y_src, y_scale, a, s)) != LAT_OK) return st;
  issue_tables(L, parent, built, s, nullptr);
  return check_launch("lattice build");
}

// The vertex lists J_v and the per-point vertex indices of a coarse level,
// built on first use (on the stream of the operator that needs them).
int ensure_lists(lattice_s* L, hipStream_t s) {
  if (L->lists_ready) return LAT_OK;
  launch_count_scan(L->table, L->vslot, &L->dc->counter, L->offsets, L->scan_work, s);
  launch_fill_lists(L->hash(), L->slot, L->rank, L->w, L->offsets, L->idx, L->entries, L->entry_w, L->chunk_first,
                    L->chunk, L->total, s);
  L->lists_ready = true;
  return check_launch("lattice lists");
}

// Table size for a build: the caller's hint, else 2 slots per point for
// the first level (surface clouds have at most about one vertex per point)
// and 2 per parent vertex for coarse levels.  A table that overflows is
// rebuilt at the worst-case size (2 slots per vertex reference) from the
// handle's own elevated positions, so no caller buffer is needed again.
int64_t initial_capacity(const lattice_s* L, const lattice_s* parent, int64_t capacity_hint) {
  const int64_t refs = 4 * L->m;
  const int64_t full = next_pow2(std::max<int64_t>(1024, 2 * refs));
  if (capacity_hint > 0) return next_pow2(std::max<int64_t>(1024, 2 * std::min(capacity_hint, refs)));
  if (parent && parent->counts_known) return std::min(full, next_pow2(std::max<int64_t>(1024, 2 * parent->n)));
  // a finest level, or a coarse one whose parent's count is not read back
  // yet: 2 slots per point (a coarse level has at most about as many
  // vertices as its parent)
  return std::min(full, next_pow2(std::max<int64_t>(1024, 2 * L->m)));
}

// The library's own stream per device (default priority) on which coarse
// levels are built, so that their construction overlaps the caller's work
// on the finer levels.  Ordering with the callers' streams:
//  - fork: a coarse build must start after the finer level's insert and
//    after every earlier use of the pool blocks it allocates from the
//    caller's stream.  When the finer level was built on the caller's
//    stream and nothing was released to that stream's pool since its
//    insert was enqueued, the side stream waits for the insert's own
//    completion event; when the finer level is side-built and nothing was
//    released since the last fork from this caller stream, no wait is
//    needed; otherwise the side stream waits for the caller's stream as it
//    is at that moment;
//  - join: before a caller's stream touches a side-built level, it waits
//    for the event that completes with that level's last build kernel.
struct SideStream {
  hipStream_t s = nullptr;
  uint64_t seq = 0;                  // side builds enqueued
  hipStream_t forked_from = nullptr; // caller stream of the last fork
  uint64_t fork_releases = 0;        // its pool's release count at that fork
  hipEvent_t ev[8] = {};             // fork / join events, used round-robin
  int next_ev = 0;
  std::vector<lattice_s*> live;      // side-built levels not yet destroyed
  hipEvent_t event() { hipEvent_t e = ev[next_ev]; next_ev = (next_ev + 1) % 8; return e; }
};
std::mutex g_side_mu;

int side_state(SideStream** out) {
  static std::map<int, SideStream*> sides;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  auto it = sides.find(dev);
  if (it == sides.end()) {
    SideStream* st = new SideStream();  // lives until exit
    HIP_TRY(hipStreamCreateWithFlags(&st->s, hipStreamNonBlocking));
    for (auto& e : st->ev) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    it = sides.emplace(dev, st).first;
  }
  *out = it->second;
  return LAT_OK;
}

// Order stream s after the side-stream build of L.
int join_side(lattice_s* L, hipStream_t s) {
  if (!L->side_seq || L->joined_by(s)) return LAT_OK;
  HIP_TRY(hipStreamWaitEvent(s, L->built, 0));
  L->joined.push_back(s);
  return LAT_OK;
}

}  // namespace

void lattice_s::free_all() {
  if (!counts_known && counts_ready) (void)hipEventSynchronize(counts_ready);
  if (side_seq && join_side(this, stream) != LAT_OK) (void)hipStreamSynchronize(bstream);
  std::vector<std::pair<void*, size_t>> bufs;
  bufs.reserve(owned.size());
  for (auto& b : owned) bufs.emplace_back(b.p, b.bytes);
  Pool::get().release_all(bufs.data(), bufs.size(), stream);
  owned.clear();
}

namespace {

// Before a handle's buffers are freed and rebuilt on its owner stream: no
// side-stream work may still read them (its own build, or that of a coarser
// level built from it).
int settle_for_rebuild(lattice_s* L) {
  SideStream* side = nullptr;
  int st;
  {
    std::lock_guard<std::mutex> lk(g_side_mu);
    if ((st = side_state(&side)) != LAT_OK) return st;
  }
  HIP_TRY(hipStreamSynchronize(side->s));
  HIP_TRY(hipStreamSynchronize(L->stream));
  return LAT_OK;
}

// Leave the side stream's bookkeeping (rebuilt on the owner stream, or
// destroyed).
void leave_side(lattice_s* L) {
  if (L->side_seq) {
    std::lock_guard<std::mutex> lk(g_side_mu);
    SideStream* side = nullptr;
    if (side_state(&side) == LAT_OK)
      side->live.erase(std::remove(side->live.begin(), side->live.end(), L), side->live.end());
  }
  L->side_seq = 0;
  L->joined.clear();
  HostSlots::get().give_event(L->built);
  L->built = nullptr;
}

// After a rebuild on the owner stream: later work there is ordered after it.
void rebuilt_on_owner_stream(lattice_s* L) { leave_side(L); }

// After a rebuild enqueued on the owner stream (from inside a call that may
// run on another stream): an event that use() makes other streams wait on.
int mark_rebuilt(lattice_s* L) {
  if (!L->rebuilt && !(L->rebuilt = HostSlots::get().take_event())) return fail(LAT_EDEVICE, "event creation failed");
  HIP_TRY(hipEventRecord(L->rebuilt, L->stream));
  L->rebuilt_joined.clear();
  return LAT_OK;
}

// Wait for a handle's counter readback; report device-side errors.
int ensure_counts(lattice_s* L) {
  if (L->counts_known) return L->status;
  if (L->parent) {
    // A coarse level is enqueued without waiting for its parent: the
    // parent's errors poison it, and a parent rebuilt after an overflow
    // (new vertex numbering) means this level is rebuilt from it as well.
    lattice_s* P = L->parent;
    const int pst = ensure_counts(P);
    if (pst != LAT_OK) {
      HIP_TRY(hipEventSynchronize(L->counts_ready));
      L->counts_known = true;
      L->status = pst;
      return fail(pst, "the lattice this one was coarsened from failed to build");
    }
    if (P->generation != L->parent_generation) {
      int st = settle_for_rebuild(L);
      if (st != LAT_OK) return st;
      L->free_all();
      rebuilt_on_owner_stream(L);
      L->parent_generation = P->generation;
      const float a[3] = {0.f, 0.f, 0.f};
      st = enqueue_build(L, nullptr, P->y, 0.5f, a, P, initial_capacity(L, P, 0), L->stream);
      if (st == LAT_OK) st = mark_rebuilt(L);
      if (st != LAT_OK) {
        L->status = st;
        return st;
      }
      ++L->generation;  // its own coarser levels were built from the old numbering
    }
  }
  HIP_TRY(hipEventSynchronize(L->counts_ready));
  if (L->m > 0 && static_cast<volatile HostCounts*>(L->host_dc)->stamp != L->stamp) {
    // the readback must belong to this build; wait for the whole stream once
    HIP_TRY(hipStreamSynchronize(L->bstream));
    if (static_cast<volatile HostCounts*>(L->host_dc)->stamp != L->stamp) {
      L->status = LAT_EDEVICE;
      return fail(LAT_EDEVICE, "vertex count readback missing after the build finished");
    }
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  L->counts_known = true;
  L->n = L->host_dc->n;
  const int dev_status = status_from_err_bits(L->host_dc->err);
  if (dev_status == LAT_EHASHFULL && L->retry_cap > L->cap) {
    // table sized from an estimate overflowed: rebuild at the worst case
    const int64_t cap = L->retry_cap;
    L->retry_cap = 0;
    int st = settle_for_rebuild(L);
    if (st != LAT_OK) return st;
    DevBuf old_y{};
    if (!L->parent) {
      for (size_t i = 0; i < L->owned.size(); ++i)
        if (L->owned[i].p == L->y) {
          old_y = L->owned[i];
          L->owned.erase(L->owned.begin() + static_cast<long>(i));
          break;
        }
    }
    L->free_all();
    rebuilt_on_owner_stream(L);
    const float a[3] = {0.f, 0.f, 0.f};
    const float* src = L->parent ? L->parent->y : static_cast<const float*>(old_y.p);
    st = enqueue_build(L, nullptr, src, L->parent ? 0.5f : 1.0f, a, L->parent, cap, L->stream);
    if (st == LAT_OK) st = mark_rebuilt(L);
    Pool::get().release(old_y.p, old_y.bytes, L->stream);
    ++L->generation;
    if (st != LAT_OK) { L->status = st; return st; }
    return ensure_counts(L);
  }
  if (dev_status != LAT_OK) {
    const char* why = dev_status == LAT_EHASHFULL ? "hash table full (raise capacity_hint)"
                      : dev_status == LAT_EKEYRANGE ? "a vertex coordinate reaches 2^20 (positions / sigma too large)"
                                                    : "non-finite position";
    L->status = dev_status;
    return fail(dev_status, why);
  }
  return LAT_OK;
}

int build_lattice(lattice_s* L, const float* pos, const float a[3], const lattice_s* parent,
                  int64_t capacity_hint, hipStream_t s, hipEvent_t built = nullptr) {
  const int64_t m = L->m;
  if (m == 0) return LAT_OK;
  if (4 * m > INT32_MAX) return fail(LAT_EUNSUPPORTED, "more than 2^29 points");
  const int64_t cap = initial_capacity(L, parent, capacity_hint);
  L->retry_cap = capacity_hint == 0 ? next_pow2(std::max<int64_t>(1024, 8 * m)) : 0;
  return enqueue_build(L, pos, parent ? parent->y : nullptr, 0.5f, a, parent, cap, s, built);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A handle not known to be poisoned; does not wait for its build.
int check_handle_nowait(const lattice_s* L) {
  if (!L) return fail(LAT_EINVAL, "null lattice handle");
  if (L->status != LAT_OK) return fail(L->status, "lattice handle is poisoned by an earlier error");
  return LAT_OK;
}

// A usable handle: not null, its vertex count read back, no device error.
int check_handle(lattice_s* L) {
  if (!L) return fail(LAT_EINVAL, "null lattice handle");
  if (L->status == LAT_OK) {
    const int st = ensure_counts(L);
    if (st != LAT_OK) return st;
  }
  if (L->status != LAT_OK) return fail(L->status, "lattice handle is poisoned by an earlier error");
  return LAT_OK;
}

// A usable handle whose device data work on stream s may read: s is ordered
// after the handle's build when that ran on the side stream.
int use(lattice_s* L, hipStream_t s) {
  int st;
  if ((st = check_handle(L)) != LAT_OK) return st;
  if (L->rebuilt && s != L->stream &&
      std::find(L->rebuilt_joined.begin(), L->rebuilt_joined.end(), s) == L->rebuilt_joined.end()) {
    // a rebuild ran on the owner stream: order this stream after it
    HIP_TRY(hipStreamWaitEvent(s, L->rebuilt, 0));
    L->rebuilt_joined.push_back(s);
  }
  return join_side(L, s);
}

// channel count / stride / alignment rules of one feature matrix
int check_matrix(const void* p, int64_t ld, int C, lat_dtype dt, const char* what, bool need_ptr) {
  const int vec = dt == LAT_BF16 ? 8 : 4;
  if (need_ptr && !p) return fail(LAT_EINVAL, std::string(what) + " is null");
  if (C <= 0) return fail(LAT_EINVAL, std::string(what) + ": channel count must be positive");
  if (C % vec != 0)
    return fail(LAT_EUNSUPPORTED, std::string(what) + ": channels must be a multiple of " + std::to_string(vec));
  if (ld < C || ld % vec != 0)
    return fail(LAT_EINVAL, std::string(what) + ": row stride must be >= channels and a multiple of " +
                                std::to_string(vec));
  if (p && !aligned16(p)) return fail(LAT_EINVAL, std::string(what) + " must be 16-byte aligned");
  return LAT_OK;
}

int check_dtype(lat_dtype dt) {
  if (dt != LAT_F32 && dt != LAT_BF16) return fail(LAT_EUNSUPPORTED, "dtype must be LAT_F32 or LAT_BF16");
  return LAT_OK;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + bbytes && y < x + abytes;
}

// Pre-activation of a convolution's input: Group Normalization over the
// input lattice's vertices, then a ReLU.
struct GnArgs {
  int groups;
  const float* gamma;
  const float* beta;
  float eps;
  const void* res;   // optional residual added to the output
  int64_t ld_res;
};

int conv_common(const int32_t* table, int64_t ldn, int64_t n_out, int64_t n_in, const void* in, int64_t ld_in,
                int Cin, const void* W, const float* bias, int Cout, lat_dtype dt, int flags,
                void* out, int64_t ld_out, const int32_t* rows, hipStream_t s, const GnArgs* gn = nullptr) {
  int st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_in == 0) ld_in = Cin;
  if (ld_out == 0) ld_out = Cout;
  if ((st = check_matrix(in, ld_in, Cin, dt, "in", n_in > 0)) != LAT_OK) return st;
  if ((st = check_matrix(out, ld_out, Cout, dt, "out", n_out > 0)) != LAT_OK) return st;
  if (!W) return fail(LAT_EINVAL, "W is null");
  if (!aligned16(W)) return fail(LAT_EINVAL, "W must be 16-byte aligned");
  if (flags & ~LAT_RELU) return fail(LAT_EINVAL, "unknown flags");
  const size_t u = dt == LAT_BF16 ? 2 : 4;
  if (n_in > 0 && n_out > 0 &&
      overlaps(in, static_cast<size_t>((n_in - 1) * ld_in + Cin) * u, out,
               static_cast<size_t>((n_out - 1) * ld_out + Cout) * u))
    return fail(LAT_EINVAL, "in and out overlap");
  if (gn) {
    if (gn->groups <= 0 || Cin % gn->groups != 0) return fail(LAT_EINVAL, "groups must divide Cin");
    if (gn->res) {
      const int64_t ld_res = gn->ld_res ? gn->ld_res : Cout;
      if ((st = check_matrix(gn->res, ld_res, Cout, dt, "res", true)) != LAT_OK) return st;
      if (n_out > 0 && overlaps(gn->res, static_cast<size_t>((n_out - 1) * ld_res + Cout) * u, out,
                                static_cast<size_t>((n_out - 1) * ld_out + Cout) * u) &&
          !(gn->res == out && ld_res == ld_out))
        return fail(LAT_EINVAL, "res and out overlap (other than res == out with the same row stride)");
    }
    if (!(gn->eps > 0.f) || !std::isfinite(gn->eps)) return fail(LAT_EINVAL, "eps must be positive and finite");
    if (Cin > conv_max_pre_channels() || Cin > gn_max_channels())
      return fail(LAT_EUNSUPPORTED, "pre-activated convolutions take at most " +
                                        std::to_string(std::min(conv_max_pre_channels(), gn_max_channels())) +
                                        " input channels");
  }
  if (n_out == 0) return LAT_OK;
  Scratch pre, work;
  if (gn) {
    // the statistics of the input lattice's rows, then the convolution
    if ((st = pre.get(sizeof(float) * 2 * static_cast<size_t>(Cin), s)) != LAT_OK) return st;
    if ((st = work.get(static_cast<size_t>(gn_workspace_bytes(n_in, Cin)), s)) != LAT_OK) return st;
    launch_gn_affine(in, ld_in, Cin, dt == LAT_BF16, n_in, gn->groups, gn->gamma, gn->beta, gn->eps,
                     pre.as<float>(), work.p, s);
  }
  launch_conv(table, ldn, n_out, n_in, in, ld_in, Cin, W, bias, Cout, dt == LAT_BF16, flags & LAT_RELU, out,
              ld_out, rows, s, gn ? pre.as<float>() : nullptr, gn ? gn->res : nullptr,
              gn && gn->res ? (gn->ld_res ? gn->ld_res : Cout) : 0);
  return check_launch("conv");
}

}  // namespace

// ---------------------------------------------------------------------------
// ABI
// ---------------------------------------------------------------------------
extern "C" {

const char* lattice_last_error(void) { return g_last_error.c_str(); }

const char* lattice_status_string(int status) {
  switch (status) {
    case LAT_OK: return "LAT_OK";
    case LAT_EINVAL: return "LAT_EINVAL";
    case LAT_EUNSUPPORTED: return "LAT_EUNSUPPORTED";
    case LAT_ENOMEM: return "LAT_ENOMEM";
    case LAT_EHASHFULL: return "LAT_EHASHFULL";
    case LAT_EKEYRANGE: return "LAT_EKEYRANGE";
    case LAT_ENONFINITE: return "LAT_ENONFINITE";
    case LAT_EDEVICE: return "LAT_EDEVICE";
    case LAT_ELEVEL: return "LAT_ELEVEL";
    default: return "LAT_UNKNOWN";
  }
}

int lattice_create(const float* pos_dev, int64_t m, int d, const float* sigma_host,
                   int64_t capacity_hint, hipStream_t stream, lattice_t* out) {
  if (!out) return fail(LAT_EINVAL, "out is null");
  *out = nullptr;
  if (d != kDim) return fail(LAT_EUNSUPPORTED, "only d = 3 is supported");
  if (m < 0) return fail(LAT_EINVAL, "m < 0");
  if (m > 0 && !pos_dev) return fail(LAT_EINVAL, "pos is null");
  if (!sigma_host) return fail(LAT_EINVAL, "sigma is null");
  if (capacity_hint < 0) return fail(LAT_EINVAL, "capacity_hint < 0");
  for (int j = 0; j < kDim; ++j)
    if (!(sigma_host[j] > 0.0f) || !std::isfinite(sigma_host[j]))
      return fail(LAT_EINVAL, "sigma must be positive and finite");
  // a_j = (d+1) sqrt(2/3) / (sigma_j sqrt((j+1)(j+2))), in double, rounded once
  float a[kDim];
  const double sc = (kDim + 1) * std::sqrt(2.0 / 3.0);
  for (int j = 0; j < kDim; ++j)
    a[j] = static_cast<float>(sc / (static_cast<double>(sigma_host[j]) *
                                    std::sqrt(static_cast<double>((j + 1) * (j + 2)))));
  lattice_s* L = new lattice_s();
  L->m = m;
  L->stream = stream;
  for (int j = 0; j < kDim; ++j) L->scale[j] = sigma_host[j];
  const int st = build_lattice(L, pos_dev, a, nullptr, capacity_hint, stream);
  if (st != LAT_OK) {
    L->free_all();
    HostSlots::get().give(L->host_dc);
    HostSlots::get().give_event(L->counts_ready);
    delete L;
    return st;
  }
  *out = L;
  return LAT_OK;
}

int lattice_create_hierarchy(const float* pos_dev, int64_t m, int d, const float* sigma_host, int levels,
                             const int64_t* capacity_hints, hipStream_t stream, lattice_t* out) {
  if (!out) return fail(LAT_EINVAL, "out is null");
  if (levels < 1 || levels > kMaxLevels)
    return fail(LAT_EINVAL, "levels must be 1 to " + std::to_string(kMaxLevels));
  for (int l = 0; l < levels; ++l) out[l] = nullptr;
  if (d != kDim) return fail(LAT_EUNSUPPORTED, "only d = 3 is supported");
  if (m < 0) return fail(LAT_EINVAL, "m < 0");
  if (m > 0 && !pos_dev) return fail(LAT_EINVAL, "pos is null");
  if (4 * m > INT32_MAX) return fail(LAT_EUNSUPPORTED, "more than 2^29 points");
  if (!sigma_host) return fail(LAT_EINVAL, "sigma is null");
  for (int j = 0; j < kDim; ++j)
    if (!(sigma_host[j] > 0.0f) || !std::isfinite(sigma_host[j]))
      return fail(LAT_EINVAL, "sigma must be positive and finite");
  float a[kDim];
  const double sc = (kDim + 1) * std::sqrt(2.0 / 3.0);
  for (int j = 0; j < kDim; ++j)
    a[j] = static_cast<float>(sc / (static_cast<double>(sigma_host[j]) *
                                    std::sqrt(static_cast<double>((j + 1) * (j + 2)))));
  lattice_s* Ls[kMaxLevels] = {};
  auto discard = [&](int st) {
    for (int l = levels - 1; l >= 0; --l) {
      if (!Ls[l]) continue;
      Ls[l]->free_all();
      HostSlots::get().give(Ls[l]->host_dc);
      HostSlots::get().give_event(Ls[l]->counts_ready);
      delete Ls[l];
    }
    return st;
  };
  // every level sized and allocated before any device work
  int st;
  for (int l = 0; l < levels; ++l) {
    lattice_s* L = new lattice_s();
    Ls[l] = L;
    L->m = m;
    L->level = l;
    L->stream = stream;
    lattice_s* parent = l ? Ls[l - 1] : nullptr;
    L->parent = parent;
    for (int j = 0; j < kDim; ++j) L->scale[j] = parent ? 2.0 * parent->scale[j] : sigma_host[j];
    if (parent) L->parent_generation = parent->generation;
    if (m == 0) continue;
    L->retry_cap = next_pow2(std::max<int64_t>(1024, 8 * m));
    const int64_t hint = capacity_hints ? std::max<int64_t>(capacity_hints[l], 0) : 0;
    if ((st = prepare_build(L, parent, initial_capacity(L, parent, hint), stream)) != LAT_OK) return discard(st);
  }
  if (m > 0) {
    // the levels' tables cleared in one launch, the inserts of all levels in
    // one launch (each level elevates the positions itself), the finest
    // level's lists, the convolution tables of all levels in one launch and
    // their row orders batched
    ClearJob jobs[kMaxLevels];
    for (int l = 0; l < levels; ++l) jobs[l] = ClearJob{Ls[l]->table, Ls[l]->cap, Ls[l]->dc, Ls[l]->scan_work};
    launch_clear_tables(jobs, levels, stream);
    InsertJob ins[kMaxLevels];
    for (int l = 0; l < levels; ++l) ins[l] = insert_job(Ls[l], pos_dev, nullptr, 1.0f, l, a);
    if ((st = issue_inserts(Ls, ins, levels, stream)) != LAT_OK) return discard(st);
    for (int l = 0; l < levels; ++l) issue_lists(Ls[l], stream);  // coarse levels: on first use
    TableJob tables[kMaxLevels];
    int64_t work_max = 0;
    for (int l = 0; l < levels; ++l) {
      int64_t work = 0;
      tables[l] = table_job(Ls[l], l ? Ls[l - 1] : nullptr, &work);
      work_max = std::max(work_max, work);
    }
    launch_level_tables(tables, levels, work_max, stream);
    RowOrderBatch batch;
    for (int l = 0; l < levels; ++l) add_row_orders(batch, Ls[l], l ? Ls[l - 1] : nullptr, stream);
    launch_row_orders(batch, nullptr, stream);
    if ((st = check_launch("lattice hierarchy build")) != LAT_OK) return discard(st);
  }
  for (int l = 0; l < levels; ++l) {
    if (l) Ls[l - 1]->children += 1;
    out[l] = Ls[l];
  }
  return LAT_OK;
}

int lattice_coarsen(lattice_t fine, int64_t capacity_hint, hipStream_t stream, lattice_t* coarse) {
  return lattice_coarsen_ex(fine, capacity_hint, 0, stream, coarse);
}

int lattice_coarsen_ex(lattice_t fine, int64_t capacity_hint, int flags, hipStream_t stream, lattice_t* coarse) {
  if (!coarse) return fail(LAT_EINVAL, "out is null");
  *coarse = nullptr;
  int st;
  if ((st = check_handle_nowait(fine)) != LAT_OK) return st;
  if (capacity_hint < 0) return fail(LAT_EINVAL, "capacity_hint < 0");
  if (flags & ~LAT_ON_STREAM) return fail(LAT_EINVAL, "unknown flags");
  lattice_s* L = new lattice_s();
  L->m = fine->m;
  L->level = fine->level + 1;
  L->parent = fine;
  for (int j = 0; j < kDim; ++j) L->scale[j] = 2.0 * fine->scale[j];
  L->parent_generation = fine->generation;
  L->stream = stream;
  const float a[3] = {0.f, 0.f, 0.f};
  // The build runs on the side stream (see SideStream), after the caller's
  // stream as it is now; callers' later work is ordered after it by use().
  SideStream* side = nullptr;
  if (L->m > 0 && !(flags & LAT_ON_STREAM)) {
    std::lock_guard<std::mutex> lk(g_side_mu);
    if ((st = side_state(&side)) != LAT_OK) {
      delete L;
      return st;
    }
    const uint64_t rel = Pool::get().release_count(stream);
    hipError_t e = hipSuccess;
    if (fine->side_seq != 0 && side->forked_from == stream && side->fork_releases == rel) {
      // ordered already: the finer level was built on the side stream
    } else if (fine->side_seq == 0 && fine->bstream == stream && fine->releases_at_insert == rel) {
      e = hipStreamWaitEvent(side->s, fine->counts_ready, 0);  // after the finer level's insert
      side->forked_from = stream;
      side->fork_releases = rel;
    } else {
      const hipEvent_t f = side->event();
      e = hipEventRecord(f, stream);
      if (e == hipSuccess) e = hipStreamWaitEvent(side->s, f, 0);
      side->forked_from = stream;
      side->fork_releases = rel;
    }
    L->built = HostSlots::get().take_event();
    if (e != hipSuccess || !L->built) {
      HostSlots::get().give_event(L->built);
      delete L;
      return fail(LAT_EDEVICE, "event record / stream wait failed");
    }
    st = build_lattice(L, nullptr, a, fine, capacity_hint, side->s, L->built);
    if (st == LAT_OK) {
      L->side_seq = ++side->seq;
      side->live.push_back(L);
    }
  } else {
    st = build_lattice(L, nullptr, a, fine, capacity_hint, stream);
  }
  if (st != LAT_OK) {
    if (side) (void)hipStreamSynchronize(side->s);
    leave_side(L);
    L->free_all();
    HostSlots::get().give(L->host_dc);
    HostSlots::get().give_event(L->counts_ready);
    delete L;
    return st;
  }
  fine->children += 1;
  *coarse = L;
  return LAT_OK;
}

int lattice_destroy(lattice_t L) {
  if (!L) return LAT_OK;
  if (L->children > 0) return fail(LAT_ELEVEL, "destroy the coarser lattices first");
  if (L->parent) L->parent->children -= 1;
  L->free_all();
  HostSlots::get().give(L->host_dc);
  HostSlots::get().give_event(L->counts_ready);
  HostSlots::get().give_event(L->rebuilt);
  leave_side(L);
  delete L;
  return LAT_OK;
}

int lattice_num_vertices(lattice_t L, int64_t* n) {
  int st;
  if (!n) return fail(LAT_EINVAL, "n is null");
  if ((st = check_handle(L)) != LAT_OK) return st;
  *n = L->n;
  return LAT_OK;
}

int lattice_num_points(lattice_t L, int64_t* m) {
  int st;
  if (!m) return fail(LAT_EINVAL, "m is null");
  if ((st = check_handle_nowait(L)) != LAT_OK) return st;
  *m = L->m;
  return LAT_OK;
}

int lattice_level(lattice_t L, int* level) {
  int st;
  if (!level) return fail(LAT_EINVAL, "level is null");
  if ((st = check_handle_nowait(L)) != LAT_OK) return st;
  *level = L->level;
  return LAT_OK;
}

int lattice_export_keys(lattice_t L, int32_t* keys_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if (L->n > 0 && !keys_dev) return fail(LAT_EINVAL, "keys is null");
  if (L->n > 0 && !aligned16(keys_dev)) return fail(LAT_EINVAL, "keys must be 16-byte aligned");
  launch_export_keys(L->vkeys, L->n, keys_dev, stream);
  return check_launch("export keys");
}

int lattice_export_simplices(lattice_t L, int32_t* idx_dev, float* w_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (L->m == 0) return LAT_OK;
  if (!idx_dev || !w_dev) return fail(LAT_EINVAL, "idx / w is null");
  HIP_TRY(hipMemcpyAsync(idx_dev, L->idx, sizeof(int32_t) * 4 * L->m, hipMemcpyDeviceToDevice, stream));
  HIP_TRY(hipMemcpyAsync(w_dev, L->w, sizeof(float) * 4 * L->m, hipMemcpyDeviceToDevice, stream));
  return LAT_OK;
}

int lattice_export_neighbors(lattice_t L, int32_t* nbr_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if (L->n == 0) return LAT_OK;
  if (!nbr_dev) return fail(LAT_EINVAL, "nbr is null");
  launch_transpose_table(L->nbr, L->nmax, L->n, nbr_dev, stream);
  return check_launch("export neighbours");
}

int lattice_conv_taps(lattice_t dst, lattice_t src, int64_t* pairs_host, hipStream_t stream) {
  int st;
  if (!pairs_host) return fail(LAT_EINVAL, "pairs is null");
  *pairs_host = 0;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  const int32_t* table;
  int64_t ld;
  if (dst == src) table = dst->nbr, ld = dst->nmax;
  else if (dst->parent == src) table = dst->down, ld = dst->nmax;
  else if (src->parent == dst) table = src->up, ld = dst->nmax;
  else return fail(LAT_ELEVEL, "dst and src must be one lattice, or one a coarsening of the other");
  if (dst->n == 0) return LAT_OK;
  Scratch cnt;
  if ((st = cnt.get(sizeof(unsigned long long), stream)) != LAT_OK) return st;
  HIP_TRY(hipMemsetAsync(cnt.p, 0, sizeof(unsigned long long), stream));
  launch_count_taps(table, ld, dst->n, cnt.as<unsigned long long>(), stream);
  if ((st = check_launch("count taps")) != LAT_OK) return st;
  unsigned long long h = 0;
  HIP_TRY(hipMemcpyAsync(&h, cnt.p, sizeof(h), hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  *pairs_host = static_cast<int64_t>(h);
  return LAT_OK;
}

int lattice_splat(lattice_t L, const void* feat_dev, int64_t ld_feat, int C, lat_dtype dt,
                  int normalize, void* vals_dev, int64_t ld_vals, float* wsum_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_feat == 0) ld_feat = C;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(feat_dev, ld_feat, C, dt, "feat", L->m > 0)) != LAT_OK) return st;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if (C > splat_max_channels(dt == LAT_BF16))
    return fail(LAT_EUNSUPPORTED, "splat supports at most " + std::to_string(splat_max_channels(dt == LAT_BF16)) +
                                      " channels");
  if (L->n == 0) return LAT_OK;
  Scratch partials;
  if ((st = partials.get(sizeof(float) * splat_partial_floats(L->total, L->chunk, C), stream)) != LAT_OK) return st;
  launch_splat(L->offsets, L->entries, L->entry_w, L->chunk_first, L->chunk, L->nmax, L->total, feat_dev, ld_feat, C,
               dt == LAT_BF16, normalize != 0, vals_dev, ld_vals, wsum_dev, partials.as<float>(), stream);
  return check_launch("splat");
}

// ---------------------------------------------------------------------------
// Splat without allocation.  Its partials live in a file-scope device array
// (each GPU holds its own copy for the life of the process).  In host code
// the array's name is only a stand-in for its device address: the address is
// looked up once per device with hipGetSymbolAddress and only that pointer
// is ever passed on.  Every call on one GPU shares the array; the splat
// writes each partial before its finishing pass reads it, so nothing needs
// clearing between calls, but calls that overlap on one GPU race.
// ---------------------------------------------------------------------------
static __device__ __align__(256) float scratch[(size_t(16) << 20) / sizeof(float)];

namespace {
constexpr size_t kNoAllocScratchBytes = sizeof(scratch);
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (looked up on the first call on
// that device).
int noalloc_scratch(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(LAT_EUNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(LAT_EDEVICE, "hipGetSymbolAddress returned no address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LAT_OK;
}
}  // namespace

int lattice_splat_noalloc(lattice_t L, const void* feat_dev, int64_t ld_feat, int C, lat_dtype dt, int normalize,
                          void* vals_dev, int64_t ld_vals, float* wsum_dev, hipStream_t stream) {
  int st;
  if (!L) return fail(LAT_EINVAL, "null lattice handle");
  if (L->status != LAT_OK) return fail(L->status, "lattice handle is poisoned by an earlier error");
  // waiting for the count may rebuild an overflowed table (an allocation):
  // the caller reads it first, as it must to size vals
  if (!L->counts_known)
    return fail(LAT_EINVAL, "read the vertex count (lattice_num_vertices) before the allocation-free splat");
  // ordered after a side-stream build without recording the join (no host
  // allocation either)
  if (L->side_seq && !L->joined_by(stream)) HIP_TRY(hipStreamWaitEvent(stream, L->built, 0));
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_feat == 0) ld_feat = C;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(feat_dev, ld_feat, C, dt, "feat", L->m > 0)) != LAT_OK) return st;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if (C > splat_max_channels(dt == LAT_BF16))
    return fail(LAT_EUNSUPPORTED, "splat supports at most " + std::to_string(splat_max_channels(dt == LAT_BF16)) +
                                      " channels");
  const size_t need = sizeof(float) * static_cast<size_t>(splat_partial_floats(L->total, L->chunk, C));
  if (need > kNoAllocScratchBytes)
    return fail(LAT_EUNSUPPORTED, "the allocation-free splat needs " + std::to_string(need) +
                                      " bytes of partials, more than its " + std::to_string(kNoAllocScratchBytes) +
                                      "-byte scratch; use lattice_splat");
  // a coarse level's lists are built in its own buffers (no allocation)
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (L->n == 0) return LAT_OK;
  void* part = nullptr;
  if ((st = noalloc_scratch(&part)) != LAT_OK) return st;
  launch_splat(L->offsets, L->entries, L->entry_w, L->chunk_first, L->chunk, L->nmax, L->total, feat_dev, ld_feat, C,
               dt == LAT_BF16, normalize != 0, vals_dev, ld_vals, wsum_dev, static_cast<float*>(part), stream);
  return check_launch("splat (no allocation)");
}

int lattice_conv(lattice_t dst, lattice_t src, const void* in_dev, int64_t ld_in, int Cin,
                 const void* W_dev, const float* bias_dev, int Cout, lat_dtype dt, int flags,
                 void* out_dev, int64_t ld_out, hipStream_t stream) {
  int st;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  const int32_t *table, *rows;
  if (dst == src) table = dst->nbr, rows = dst->nbr_rows;
  else if (dst->parent == src) table = dst->down, rows = dst->down_rows;
  else return fail(LAT_ELEVEL, "dst must be src or lattice_coarsen(src)");
  return conv_common(table, dst->nmax, dst->n, src->n, in_dev, ld_in, Cin, W_dev, bias_dev, Cout, dt, flags,
                     out_dev, ld_out, rows, stream);
}

int lattice_refine(lattice_t fine, lattice_t coarse, const void* in_dev, int64_t ld_in, int Cin,
                   const void* W_dev, const float* bias_dev, int Cout, lat_dtype dt, int flags,
                   void* out_dev, int64_t ld_out, hipStream_t stream) {
  int st;
  if ((st = use(fine, stream)) != LAT_OK) return st;
  if ((st = use(coarse, stream)) != LAT_OK) return st;
  if (coarse->parent != fine) return fail(LAT_ELEVEL, "coarse must be lattice_coarsen(fine)");
  return conv_common(coarse->up, fine->nmax, fine->n, coarse->n, in_dev, ld_in, Cin, W_dev, bias_dev, Cout, dt,
                     flags, out_dev, ld_out, coarse->up_rows, stream);
}

int lattice_conv_preact(lattice_t dst, lattice_t src, const void* in_dev, int64_t ld_in, int Cin, int groups,
                        const float* gamma_dev, const float* beta_dev, float eps, const void* W_dev,
                        const float* bias_dev, int Cout, lat_dtype dt, int flags, const void* res_dev,
                        int64_t ld_res, void* out_dev, int64_t ld_out, hipStream_t stream) {
  int st;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  const int32_t *table, *rows;
  if (dst == src) table = dst->nbr, rows = dst->nbr_rows;
  else if (dst->parent == src) table = dst->down, rows = dst->down_rows;
  else return fail(LAT_ELEVEL, "dst must be src or lattice_coarsen(src)");
  const GnArgs gn{groups, gamma_dev, beta_dev, eps, res_dev, ld_res};
  return conv_common(table, dst->nmax, dst->n, src->n, in_dev, ld_in, Cin, W_dev, bias_dev, Cout, dt, flags,
                     out_dev, ld_out, rows, stream, &gn);
}

int lattice_refine_preact(lattice_t fine, lattice_t coarse, const void* in_dev, int64_t ld_in, int Cin, int groups,
                          const float* gamma_dev, const float* beta_dev, float eps, const void* W_dev,
                          const float* bias_dev, int Cout, lat_dtype dt, int flags, void* out_dev, int64_t ld_out,
                          hipStream_t stream) {
  int st;
  if ((st = use(fine, stream)) != LAT_OK) return st;
  if ((st = use(coarse, stream)) != LAT_OK) return st;
  if (coarse->parent != fine) return fail(LAT_ELEVEL, "coarse must be lattice_coarsen(fine)");
  const GnArgs gn{groups, gamma_dev, beta_dev, eps, nullptr, 0};
  return conv_common(coarse->up, fine->nmax, fine->n, coarse->n, in_dev, ld_in, Cin, W_dev, bias_dev, Cout, dt,
                     flags, out_dev, ld_out, coarse->up_rows, stream, &gn);
}

int lattice_distribute_pointnet(lattice_t L, const float* pos_dev, const float* feat_dev, int64_t ld_feat,
                                int Cf, const float* gn_gamma_dev, const float* gn_beta_dev, float eps,
                                const float* W1_dev, const float* b1_dev, int C1, const float* W2_dev,
                                const float* b2_dev, int C2, const float* W3_dev, const float* b3_dev, int C3,
                                lat_dtype out_dt, void* out_dev, int64_t ld_out, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (Cf < 0 || Cf > distribute_max_features())
    return fail(LAT_EUNSUPPORTED, "Cf must be in [0, " + std::to_string(distribute_max_features()) + "]");
  for (int c : {C1, C2, C3})
    if (c <= 0 || c % 16 != 0 || c > 64) return fail(LAT_EUNSUPPORTED, "C1, C2, C3 must be 16, 32, 48 or 64");
  if (C1 == 48 || C2 == 48)
    return fail(LAT_EUNSUPPORTED, "a normalised layer input of 48 channels does not split into 32 groups");
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(LAT_EINVAL, "eps must be finite and >= 0");
  if (ld_feat == 0) ld_feat = Cf;
  if (ld_out == 0) ld_out = C3;
  if (ld_feat < Cf) return fail(LAT_EINVAL, "ld_feat < Cf");
  if ((st = check_dtype(out_dt)) != LAT_OK) return st;
  if ((st = check_matrix(out_dev, ld_out, C3, out_dt, "out", L->n > 0)) != LAT_OK) return st;
  if (!W1_dev || !W2_dev || !W3_dev) return fail(LAT_EINVAL, "weights are null");
  if (L->m > 0 && !pos_dev) return fail(LAT_EINVAL, "pos is null");
  if (L->m > 0 && Cf > 0 && !feat_dev) return fail(LAT_EINVAL, "feat is null");
  if (L->n > 0 && !out_dev) return fail(LAT_EINVAL, "out is null");
  if (L->n == 0) return LAT_OK;
  Scratch work;
  const int bf = out_dt == LAT_BF16;
  if ((st = work.get(static_cast<size_t>(distribute_workspace_bytes(L->n, L->total, C3, bf)), stream)) != LAT_OK)
    return st;
  launch_distribute(L->offsets, L->entries, L->chunk_first, L->chunk, L->n, L->total, pos_dev, L->scale, feat_dev,
                    ld_feat, Cf, gn_gamma_dev, gn_beta_dev, eps, W1_dev, b1_dev, C1, W2_dev, b2_dev, C2, W3_dev,
                    b3_dev, C3, out_dev, bf, ld_out, work.p, stream);
  return check_launch("distribute");
}

int lattice_slice(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                  float* out_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(out_dev, C, C, LAT_F32, "out", L->m > 0)) != LAT_OK) return st;
  launch_slice(L->idx, L->w, L->m, vals_dev, ld_vals, C, dt == LAT_BF16, out_dev, stream);
  return check_launch("slice");
}

int lattice_deform_slice(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                         const float* wv_dev, float beta, float* out_dev, float* delta_dev,
                         hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(out_dev, C, C, LAT_F32, "out", L->m > 0)) != LAT_OK) return st;
  if (!wv_dev) return fail(LAT_EINVAL, "wv is null");
  if (!std::isfinite(beta)) return fail(LAT_EINVAL, "beta must be finite");
  if (delta_dev && !aligned16(delta_dev)) return fail(LAT_EINVAL, "delta must be 16-byte aligned");
  if (C > deform_max_channels(dt == LAT_BF16))
    return fail(LAT_EUNSUPPORTED, "DeformSlice supports at most " +
                                      std::to_string(deform_max_channels(dt == LAT_BF16)) + " channels");
  launch_deform_slice(L->idx, L->w, L->m, vals_dev, ld_vals, C, dt == LAT_BF16, wv_dev, beta, out_dev,
                      delta_dev, nullptr, stream);
  return check_launch("deform slice");
}

int lattice_slice_and_deform(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                             const float* wv_dev, float beta, float* slice_dev, float* deform_dev,
                             hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(slice_dev, C, C, LAT_F32, "slice_out", L->m > 0)) != LAT_OK) return st;
  if ((st = check_matrix(deform_dev, C, C, LAT_F32, "deform_out", L->m > 0)) != LAT_OK) return st;
  if (L->m > 0 && overlaps(slice_dev, sizeof(float) * static_cast<size_t>(L->m) * C, deform_dev,
                           sizeof(float) * static_cast<size_t>(L->m) * C))
    return fail(LAT_EINVAL, "slice_out and deform_out overlap");
  if (!wv_dev) return fail(LAT_EINVAL, "wv is null");
  if (!std::isfinite(beta)) return fail(LAT_EINVAL, "beta must be finite");
  if (C > deform_max_channels(dt == LAT_BF16))
    return fail(LAT_EUNSUPPORTED, "DeformSlice supports at most " +
                                      std::to_string(deform_max_channels(dt == LAT_BF16)) + " channels");
  launch_deform_slice(L->idx, L->w, L->m, vals_dev, ld_vals, C, dt == LAT_BF16, wv_dev, beta, deform_dev,
                      nullptr, slice_dev, stream);
  return check_launch("slice and deform slice");
}

int lattice_deform_slice_classify(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                                  const float* wv_dev, float beta, const float* Wc_dev, const float* bc_dev, int K,
                                  float* logits_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if ((st = check_matrix(vals_dev, ld_vals, C, dt, "vals", L->n > 0)) != LAT_OK) return st;
  if (!wv_dev || !Wc_dev) return fail(LAT_EINVAL, "wv and Wc must not be null");
  if (L->m > 0 && !logits_dev) return fail(LAT_EINVAL, "logits is null");
  if (!std::isfinite(beta)) return fail(LAT_EINVAL, "beta must be finite");
  if (K <= 0 || K > deform_classify_max_classes())
    return fail(LAT_EUNSUPPORTED, "K must be in [1, " + std::to_string(deform_classify_max_classes()) + "]");
  if (C > deform_max_channels(dt == LAT_BF16) || static_cast<int64_t>(K) * C > deform_classify_max_weights())
    return fail(LAT_EUNSUPPORTED, "the classifier takes at most " + std::to_string(deform_classify_max_weights()) +
                                      " weights (K x C) and DeformSlice's channel limit");
  if (!aligned16(Wc_dev)) return fail(LAT_EINVAL, "Wc must be 16-byte aligned");
  launch_deform_classify(L->idx, L->w, L->m, vals_dev, ld_vals, C, dt == LAT_BF16, wv_dev, beta, Wc_dev, bc_dev, K,
                         logits_dev, stream);
  return check_launch("deform slice classify");
}

// ---- backward passes ----

int lattice_splat_backward(lattice_t L, const float* dX_dev, int64_t ld_dX, int C, int normalize,
                           const float* wsum_dev, float* dF_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (ld_dX == 0) ld_dX = C;
  if ((st = check_matrix(dX_dev, ld_dX, C, LAT_F32, "dX", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(dF_dev, C, C, LAT_F32, "dF", L->m > 0)) != LAT_OK) return st;
  if (L->m == 0) return LAT_OK;
  ScopedKernelTimer tm("splat_bwd", stream);
  const float* src = dX_dev;
  int64_t ld = ld_dX;
  Scratch scaled;
  if (normalize) {
    if ((st = scaled.get(sizeof(float) * static_cast<size_t>(L->n) * C, stream)) != LAT_OK) return st;
    launch_scale_by_weight_sum(L->offsets, L->entry_w, wsum_dev, L->n, dX_dev, ld_dX, C, scaled.as<float>(), C,
                               stream);
    src = scaled.as<float>();
    ld = C;
  }
  launch_slice(L->idx, L->w, L->m, src, ld, C, false, dF_dev, stream);
  return check_launch("splat backward");
}

int lattice_slice_backward(lattice_t L, const float* dOut_dev, int64_t ld_dOut, int C, float* dX_dev, int64_t ld_dX,
                           hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (ld_dOut == 0) ld_dOut = C;
  if (ld_dX == 0) ld_dX = C;
  if ((st = check_matrix(dOut_dev, ld_dOut, C, LAT_F32, "dOut", L->m > 0)) != LAT_OK) return st;
  if ((st = check_matrix(dX_dev, ld_dX, C, LAT_F32, "dX", L->n > 0)) != LAT_OK) return st;
  if (C > splat_max_channels(false))
    return fail(LAT_EUNSUPPORTED, "slice backward supports at most " + std::to_string(splat_max_channels(false)) +
                                      " channels");
  if (L->n == 0) return LAT_OK;
  ScopedKernelTimer tm("slice_bwd", stream);
  Scratch partials;
  if ((st = partials.get(sizeof(float) * splat_partial_floats(L->total, L->chunk, C), stream)) != LAT_OK) return st;
  launch_splat(L->offsets, L->entries, L->entry_w, L->chunk_first, L->chunk, L->nmax, L->total, dOut_dev, ld_dOut, C,
               false, false, dX_dev, ld_dX, nullptr, partials.as<float>(), stream);
  return check_launch("slice backward");
}

namespace {

// The body of lattice_conv_backward once both lattices are in use on stream.
int conv_backward_impl(lattice_t dst, lattice_t src, const void* X_dev, int64_t ld_X, int Cin, const void* W_dev,
                       int Cout, lat_dtype dt, int flags, const void* Y_dev, int64_t ld_Y, const void* dY_dev,
                       int64_t ld_dY, void* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev,
                       hipStream_t stream) {
  int st;
  if ((st = check_dtype(dt)) != LAT_OK) return st;
  const bool bf = dt == LAT_BF16;
  const size_t u = bf ? 2 : 4;
  // the forward's table (dst rows, src values) and the adjoint's (src rows,
  // dst values)
  const int32_t *fwd, *adj, *adj_rows = nullptr;
  int64_t fwd_ld, adj_ld;
  if (dst == src) {
    fwd = adj = dst->nbr;
    fwd_ld = adj_ld = dst->nmax;
    adj_rows = dst->nbr_rows;
  } else if (dst->parent == src) {            // strided: adjoint is the Upsample into src
    fwd = dst->down;
    fwd_ld = dst->nmax;
    adj = dst->up;
    adj_ld = src->nmax;
    adj_rows = dst->up_rows;
  } else if (src->parent == dst) {            // Upsample into dst: adjoint is the strided conv
    fwd = src->up;
    fwd_ld = dst->nmax;
    adj = src->down;
    adj_ld = src->nmax;
    adj_rows = src->down_rows;
  } else {
    return fail(LAT_ELEVEL, "dst and src must be one lattice, or one a coarsening of the other");
  }
  if (flags & ~LAT_RELU) return fail(LAT_EINVAL, "unknown flags");
  const bool relu = (flags & LAT_RELU) != 0;
  if (ld_dY == 0) ld_dY = Cout;
  if (ld_Y == 0) ld_Y = Cout;
  if (ld_X == 0) ld_X = Cin;
  if (ld_dX == 0) ld_dX = Cin;
  const int64_t n_out = dst->n, n_in = src->n;
  if ((st = check_matrix(dY_dev, ld_dY, Cout, dt, "dY", n_out > 0)) != LAT_OK) return st;
  if (relu && (st = check_matrix(Y_dev, ld_Y, Cout, dt, "Y", n_out > 0)) != LAT_OK) return st;
  if (dX_dev) {
    if ((st = check_matrix(dX_dev, ld_dX, Cin, dt, "dX", false)) != LAT_OK) return st;
    if (!W_dev) return fail(LAT_EINVAL, "W is null");
    if (!aligned16(W_dev)) return fail(LAT_EINVAL, "W must be 16-byte aligned");
    if (n_in > 0 && n_out > 0 &&
        overlaps(dX_dev, u * static_cast<size_t>((n_in - 1) * ld_dX + Cin), dY_dev,
                 u * static_cast<size_t>((n_out - 1) * ld_dY + Cout)))
      return fail(LAT_EINVAL, "dX and dY overlap");
  }
  if (dW_dev || dbias_dev) {
    if ((st = check_matrix(X_dev, ld_X, Cin, dt, "X", dW_dev != nullptr && n_in > 0)) != LAT_OK) return st;
    if (dW_dev && !aligned16(dW_dev)) return fail(LAT_EINVAL, "dW must be 16-byte aligned");
    if (dbias_dev && !aligned16(dbias_dev)) return fail(LAT_EINVAL, "dbias must be 16-byte aligned");
  }
  if (!dX_dev && !dW_dev && !dbias_dev) return LAT_OK;
  ScopedKernelTimer tm("conv_bwd", stream);
  const void* G = dY_dev;
  int64_t ld_G = ld_dY;
  Scratch masked, wt, partials;
  const bool need_mask = relu && n_out > 0, need_wt = dX_dev && n_in > 0;
  if (need_mask && (st = masked.get(u * static_cast<size_t>(n_out) * Cout, stream)) != LAT_OK) return st;
  if (need_wt && (st = wt.get(u * 9 * static_cast<size_t>(Cin) * Cout, stream)) != LAT_OK) return st;
  launch_conv_bwd_prep(dY_dev, ld_dY, Y_dev, ld_Y, n_out, need_mask ? masked.p : nullptr, Cout, W_dev, Cout, Cin,
                       need_wt ? wt.p : nullptr, bf ? 1 : 0, stream);
  if (need_mask) {
    G = masked.p;
    ld_G = Cout;
  }
  if (need_wt) {
    launch_conv(adj, adj_ld, n_in, n_out, G, ld_G, Cout, wt.p, nullptr, Cin, bf ? 1 : 0, false, dX_dev, ld_dX,
                adj_rows, stream);
  }
  if (dW_dev || dbias_dev) {
    const int64_t pf = wgrad_partial_floats(n_out, Cout, Cin);
    if (pf > 0 && (st = partials.get(sizeof(float) * static_cast<size_t>(pf), stream)) != LAT_OK) return st;
    launch_conv_wgrad(fwd, fwd_ld, n_out, X_dev, ld_X, Cin, G, ld_G, Cout, dW_dev, dbias_dev, partials.as<float>(),
                      bf ? 1 : 0, stream);
  }
  return check_launch("conv backward");
}

}  // namespace

int lattice_conv_backward(lattice_t dst, lattice_t src, const float* X_dev, int64_t ld_X, int Cin, const float* W_dev,
                          int Cout, int flags, const float* Y_dev, int64_t ld_Y, const float* dY_dev, int64_t ld_dY,
                          float* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev, hipStream_t stream) {
  int st;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  return conv_backward_impl(dst, src, X_dev, ld_X, Cin, W_dev, Cout, LAT_F32, flags, Y_dev, ld_Y, dY_dev, ld_dY,
                            dX_dev, ld_dX, dW_dev, dbias_dev, stream);
}

int lattice_conv_backward_ex(lattice_t dst, lattice_t src, const void* X_dev, int64_t ld_X, int Cin, const void* W_dev,
                             int Cout, lat_dtype dt, int flags, const void* Y_dev, int64_t ld_Y, const void* dY_dev,
                             int64_t ld_dY, void* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev,
                             hipStream_t stream) {
  int st;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  return conv_backward_impl(dst, src, X_dev, ld_X, Cin, W_dev, Cout, dt, flags, Y_dev, ld_Y, dY_dev, ld_dY, dX_dev,
                            ld_dX, dW_dev, dbias_dev, stream);
}

int lattice_conv_preact_backward(lattice_t dst, lattice_t src, const float* X_dev, int64_t ld_X, int Cin, int groups,
                                 const float* gamma_dev, const float* beta_dev, float eps, const float* W_dev,
                                 int Cout, int flags, const float* Y_dev, int64_t ld_Y, const float* dY_dev,
                                 int64_t ld_dY, float* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev,
                                 float* dgamma_dev, float* dbeta_dev, hipStream_t stream) {
  int st;
  if ((st = use(dst, stream)) != LAT_OK) return st;
  if ((st = use(src, stream)) != LAT_OK) return st;
  if (!(dst == src || dst->parent == src || src->parent == dst))
    return fail(LAT_ELEVEL, "dst and src must be one lattice, or one a coarsening of the other");
  if (groups <= 0 || Cin % groups != 0) return fail(LAT_EINVAL, "groups must divide Cin");
  if (!(eps > 0.f) || !std::isfinite(eps)) return fail(LAT_EINVAL, "eps must be positive and finite");
  if (Cin > gn_max_channels())
    return fail(LAT_EUNSUPPORTED, "the pre-activated convolution's backward takes at most " +
                                      std::to_string(gn_max_channels()) + " input channels");
  if (ld_X == 0) ld_X = Cin;
  if (ld_dX == 0) ld_dX = Cin;
  const int64_t n_in = src->n;
  if ((st = check_matrix(X_dev, ld_X, Cin, LAT_F32, "X", n_in > 0)) != LAT_OK) return st;
  if (dX_dev) {
    if ((st = check_matrix(dX_dev, ld_dX, Cin, LAT_F32, "dX", n_in > 0)) != LAT_OK) return st;
    if (n_in > 0 && overlaps(dX_dev, sizeof(float) * static_cast<size_t>((n_in - 1) * ld_dX + Cin), X_dev,
                             sizeof(float) * static_cast<size_t>((n_in - 1) * ld_X + Cin)))
      return fail(LAT_EINVAL, "dX and X overlap");
  }
  const bool need_dA = dX_dev || dgamma_dev || dbeta_dev;
  if (!need_dA && !dW_dev && !dbias_dev) return LAT_OK;
  const size_t nc = static_cast<size_t>(n_in) * Cin;
  Scratch pre, stats, work, act, dact, coef;
  if ((st = pre.get(sizeof(float) * 2 * static_cast<size_t>(Cin), stream)) != LAT_OK) return st;
  if ((st = stats.get(sizeof(double) * 2 * static_cast<size_t>(groups), stream)) != LAT_OK) return st;
  if ((st = work.get(static_cast<size_t>(gn_workspace_bytes(n_in, Cin)), stream)) != LAT_OK) return st;
  if ((st = act.get(sizeof(float) * std::max<size_t>(nc, 4), stream)) != LAT_OK) return st;
  if (need_dA && (st = dact.get(sizeof(float) * std::max<size_t>(nc, 4), stream)) != LAT_OK) return st;
  if ((st = coef.get(sizeof(float) * 4 * static_cast<size_t>(Cin), stream)) != LAT_OK) return st;
  // the forward's pre-activated input, then the convolution's backward on it
  launch_gn_affine(X_dev, ld_X, Cin, 0, n_in, groups, gamma_dev, beta_dev, eps, pre.as<float>(), work.p, stream,
                   stats.as<double>());
  launch_gn_relu_apply(X_dev, ld_X, Cin, n_in, pre.as<float>(), act.as<float>(), Cin, stream);
  if ((st = conv_backward_impl(dst, src, act.as<float>(), Cin, Cin, W_dev, Cout, LAT_F32, flags, Y_dev, ld_Y, dY_dev,
                               ld_dY, need_dA ? dact.as<float>() : nullptr, Cin, dW_dev, dbias_dev, stream)) != LAT_OK)
    return st;
  if (need_dA)
    launch_gn_backward(X_dev, ld_X, dact.as<float>(), Cin, Cin, groups, n_in, gamma_dev, pre.as<float>(),
                       stats.as<double>(), dgamma_dev, dbeta_dev, coef.as<float>(), dX_dev, ld_dX, work.p, stream);
  return check_launch("pre-activated conv backward");
}

int lattice_deform_slice_backward(lattice_t L, const float* vals_dev, int64_t ld_vals, int C, const float* wv_dev,
                                  float beta, const float* dOut_dev, int64_t ld_dOut, float* dvals_dev,
                                  int64_t ld_dvals, float* dwv_dev, float* dbeta_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if (ld_dOut == 0) ld_dOut = C;
  if (ld_dvals == 0) ld_dvals = C;
  if ((st = check_matrix(vals_dev, ld_vals, C, LAT_F32, "vals", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(dOut_dev, ld_dOut, C, LAT_F32, "dOut", L->m > 0)) != LAT_OK) return st;
  if ((st = check_matrix(dvals_dev, ld_dvals, C, LAT_F32, "dvals", L->n > 0)) != LAT_OK) return st;
  if (!wv_dev || !dwv_dev || !dbeta_dev) return fail(LAT_EINVAL, "wv, dwv and dbeta must not be null");
  if (!std::isfinite(beta)) return fail(LAT_EINVAL, "beta must be finite");
  if (C > deform_max_channels(false))
    return fail(LAT_EUNSUPPORTED, "DeformSlice backward supports at most " +
                                      std::to_string(deform_max_channels(false)) + " channels");
  if (L->n > 0 &&
      overlaps(dvals_dev, sizeof(float) * static_cast<size_t>((L->n - 1) * ld_dvals + C), vals_dev,
               sizeof(float) * static_cast<size_t>((L->n - 1) * ld_vals + C)))
    return fail(LAT_EINVAL, "dvals and vals overlap");
  Scratch work;
  if ((st = work.get(static_cast<size_t>(deform_backward_workspace_bytes(L->m, C, L->total, L->chunk)), stream)) !=
      LAT_OK)
    return st;
  launch_deform_slice_backward(L->idx, L->w, L->m, L->offsets, L->entries, L->chunk_first, L->chunk, L->nmax,
                               L->total, vals_dev, ld_vals, C, wv_dev, beta, dOut_dev, ld_dOut, dvals_dev, ld_dvals,
                               dwv_dev, dbeta_dev, work.p, stream);
  return check_launch("deform slice backward");
}

int lattice_deform_slice_classify_backward(lattice_t L, const float* vals_dev, int64_t ld_vals, int C,
                                           const float* wv_dev, float beta, const float* Wc_dev, int K,
                                           const float* dlogits_dev, int64_t ld_dlogits, float* dvals_dev,
                                           int64_t ld_dvals, float* dwv_dev, float* dbeta_dev, float* dWc_dev,
                                           float* dbc_dev, hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (ld_vals == 0) ld_vals = C;
  if (ld_dvals == 0) ld_dvals = C;
  if (ld_dlogits == 0) ld_dlogits = K;
  if ((st = check_matrix(vals_dev, ld_vals, C, LAT_F32, "vals", L->n > 0)) != LAT_OK) return st;
  if ((st = check_matrix(dvals_dev, ld_dvals, C, LAT_F32, "dvals", L->n > 0)) != LAT_OK) return st;
  if (!wv_dev || !Wc_dev || !dwv_dev || !dbeta_dev) return fail(LAT_EINVAL, "wv, Wc, dwv and dbeta must not be null");
  if (L->m > 0 && !dlogits_dev) return fail(LAT_EINVAL, "dlogits is null");
  if (!std::isfinite(beta)) return fail(LAT_EINVAL, "beta must be finite");
  if (K <= 0 || K > deform_classify_max_classes())
    return fail(LAT_EUNSUPPORTED, "K must be in [1, " + std::to_string(deform_classify_max_classes()) + "]");
  if (ld_dlogits < K) return fail(LAT_EINVAL, "ld_dlogits < K");
  if (C > deform_max_channels(false) || static_cast<int64_t>(K) * C > deform_classify_max_weights())
    return fail(LAT_EUNSUPPORTED, "the classifier takes at most " + std::to_string(deform_classify_max_weights()) +
                                      " weights (K x C) and DeformSlice's channel limit");
  if (!aligned16(Wc_dev)) return fail(LAT_EINVAL, "Wc must be 16-byte aligned");
  if (L->n > 0 &&
      overlaps(dvals_dev, sizeof(float) * static_cast<size_t>((L->n - 1) * ld_dvals + C), vals_dev,
               sizeof(float) * static_cast<size_t>((L->n - 1) * ld_vals + C)))
    return fail(LAT_EINVAL, "dvals and vals overlap");
  const size_t mc = std::max<size_t>(static_cast<size_t>(L->m) * C, 4);
  Scratch feat, dfeat, part, work;
  if ((st = feat.get(sizeof(float) * mc, stream)) != LAT_OK) return st;
  if ((st = dfeat.get(sizeof(float) * mc, stream)) != LAT_OK) return st;
  if ((st = part.get(sizeof(float) * static_cast<size_t>(classify_backward_partial_floats(L->m, K, C)), stream)) !=
      LAT_OK)
    return st;
  if ((st = work.get(static_cast<size_t>(deform_backward_workspace_bytes(L->m, C, L->total, L->chunk)), stream)) !=
      LAT_OK)
    return st;
  // the forward's per-point features, then their gradient and the classifier's
  launch_deform_slice(L->idx, L->w, L->m, vals_dev, ld_vals, C, 0, wv_dev, beta, feat.as<float>(), nullptr, nullptr,
                      stream);
  launch_classify_backward(dlogits_dev, ld_dlogits, Wc_dev, K, C, L->m, feat.as<float>(), dfeat.as<float>(), dWc_dev,
                           dbc_dev, part.as<float>(), stream);
  launch_deform_slice_backward(L->idx, L->w, L->m, L->offsets, L->entries, L->chunk_first, L->chunk, L->nmax,
                               L->total, vals_dev, ld_vals, C, wv_dev, beta, dfeat.as<float>(), C, dvals_dev,
                               ld_dvals, dwv_dev, dbeta_dev, work.p, stream);
  return check_launch("deform slice classify backward");
}

int lattice_distribute_pointnet_backward(lattice_t L, const float* pos_dev, const float* feat_dev, int64_t ld_feat,
                                         int Cf, const float* gn_gamma_dev, const float* gn_beta_dev, float eps,
                                         const float* W1_dev, const float* b1_dev, int C1, const float* W2_dev,
                                         const float* b2_dev, int C2, const float* W3_dev, const float* b3_dev, int C3,
                                         const float* dX_dev, int64_t ld_dX, float* dfeat_dev, int64_t ld_dfeat,
                                         float* dW1_dev, float* db1_dev, float* dW2_dev, float* db2_dev,
                                         float* dW3_dev, float* db3_dev, float* dgamma_dev, float* dbeta_dev,
                                         hipStream_t stream) {
  int st;
  if ((st = use(L, stream)) != LAT_OK) return st;
  if ((st = ensure_lists(L, stream)) != LAT_OK) return st;
  if (Cf < 0 || Cf > distribute_max_features())
    return fail(LAT_EUNSUPPORTED, "Cf must be in [0, " + std::to_string(distribute_max_features()) + "]");
  for (int c : {C1, C2, C3})
    if (c <= 0 || c % 16 != 0 || c > 64) return fail(LAT_EUNSUPPORTED, "C1, C2, C3 must be 16, 32, 48 or 64");
  if (C1 == 48 || C2 == 48)
    return fail(LAT_EUNSUPPORTED, "a normalised layer input of 48 channels does not split into 32 groups");
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(LAT_EINVAL, "eps must be finite and >= 0");
  if (ld_feat == 0) ld_feat = Cf;
  if (ld_dfeat == 0) ld_dfeat = Cf;
  if (ld_dX == 0) ld_dX = C3;
  if (ld_feat < Cf || ld_dfeat < Cf) return fail(LAT_EINVAL, "feature row strides must be >= Cf");
  if ((st = check_matrix(dX_dev, ld_dX, C3, LAT_F32, "dX", L->n > 0)) != LAT_OK) return st;
  if (!W1_dev || !W2_dev || !W3_dev) return fail(LAT_EINVAL, "weights are null");
  if (!aligned16(W2_dev) || !aligned16(W3_dev)) return fail(LAT_EINVAL, "W2 and W3 must be 16-byte aligned");
  if (L->m > 0 && !pos_dev) return fail(LAT_EINVAL, "pos is null");
  if (L->m > 0 && Cf > 0 && !feat_dev) return fail(LAT_EINVAL, "feat is null");
  Scratch work;
  if ((st = work.get(static_cast<size_t>(distribute_backward_workspace_bytes(L->n, L->m, L->total, Cf, C1, C2, C3)),
                     stream)) != LAT_OK)
    return st;
  launch_distribute_backward(L->offsets, L->entries, L->chunk_first, L->chunk, L->n, L->m, L->total, pos_dev,
                             L->scale, feat_dev, ld_feat, Cf, gn_gamma_dev, gn_beta_dev, eps, W1_dev, b1_dev, C1,
                             W2_dev, b2_dev, C2, W3_dev, b3_dev, C3, dX_dev, ld_dX, dfeat_dev, ld_dfeat, dW1_dev,
                             db1_dev, dW2_dev, db2_dev, dW3_dev, db3_dev, dgamma_dev, dbeta_dev, work.p, stream);
  return check_launch("distribute backward");
}

int lattice_timing_enable(const char* name, int enable) {
  if (!name) return fail(LAT_EINVAL, "name is null");
  std::lock_guard<std::mutex> lk(g_timer_mu);
  TimerFamily* f = find_family(name, true);
  f->enabled = enable != 0;
  g_any_timer = false;
  for (auto& fam : timer_families()) g_any_timer = g_any_timer || fam.enabled;
  return LAT_OK;
}

int lattice_timing_read(const char* name, int64_t* launches, double* total_ms) {
  if (!name || !launches || !total_ms) return fail(LAT_EINVAL, "null argument");
  std::lock_guard<std::mutex> lk(g_timer_mu);
  *launches = 0;
  *total_ms = 0.0;
  TimerFamily* f = find_family(name, false);
  if (!f) return LAT_OK;
  for (auto& pr : f->recorded) {
    HIP_TRY(hipEventSynchronize(pr.second));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, pr.first, pr.second));
    *total_ms += ms;
    *launches += 1;
    f->spare.push_back(pr.first);
    f->spare.push_back(pr.second);
  }
  f->recorded.clear();
  return LAT_OK;
}

}  // extern "C"

// C ABI of the PSS layer: argument checks, parameter set-up, dispatch and the
// library-owned scratch pool.  Every check runs on the host before anything
// is enqueued.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <map>
#include <mutex>

#include "../../include/pss.h"
#include "pss_launch.hpp"

namespace {

using pss::KParams;

// Bags and items are indexed with 32-bit integers in the sorted deposit.
constexpr uint64_t kMaxBags = (1ull << 32) - 1;
constexpr int64_t kMaxItems = (1ll << 32) - 1;

int check_common(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hp) {
  if (hp == nullptr) return PSS_ERR_INVALID_ARG;
  if (M < 1 || M > static_cast<int64_t>(PSS_PRIME)) return PSS_ERR_INVALID_ARG;
  if (Z < 1 || static_cast<int64_t>(Z) > M) return PSS_ERR_INVALID_ARG;
  if (d < 1 || d > PSS_MAX_DIM || d % Z != 0) return PSS_ERR_INVALID_ARG;
  if (hp->a < 1 || hp->a > PSS_PRIME - 1) return PSS_ERR_INVALID_ARG;
  if (hp->b > PSS_PRIME - 1) return PSS_ERR_INVALID_ARG;
  if (hp->num_tables < 1 || hp->batch < 1) return PSS_ERR_INVALID_ARG;
  const uint64_t bags = static_cast<uint64_t>(hp->num_tables) * hp->batch;
  if (bags > kMaxBags) return PSS_ERR_INVALID_ARG;
  const uint64_t TC = static_cast<uint64_t>(hp->num_tables) * static_cast<uint64_t>(d / Z);
  if (TC >= (1ull << 32)) return PSS_ERR_INVALID_ARG;
  if (hp->num_indices < 0 || hp->num_indices > kMaxItems) return PSS_ERR_INVALID_ARG;
  if (hp->weight_dtype != PSS_F32 && hp->weight_dtype != PSS_BF16) return PSS_ERR_UNSUPPORTED;
  if (hp->flags & ~PSS_FLAGS_ALL) return PSS_ERR_INVALID_ARG;
  if ((hp->flags & PSS_SIGN_MASK) == PSS_SIGN_MASK) return PSS_ERR_INVALID_ARG;
  if (hp->flags & PSS_SIGN_MASK) {
    if (hp->sign_a < 1 || hp->sign_a > PSS_PRIME - 1) return PSS_ERR_INVALID_ARG;
    if (hp->sign_b > PSS_PRIME - 1) return PSS_ERR_INVALID_ARG;
  }
  // int32 offsets cannot describe more than 2^31 - 1 items
  if ((hp->flags & PSS_INDEX_I32) && hp->num_indices > INT32_MAX) return PSS_ERR_INVALID_ARG;
  return PSS_OK;
}

KParams make_params(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hp) {
  KParams p;
  const pss::FastMod fm = pss::make_fastmod(static_cast<uint32_t>(M));
  p.fm_c = fm.c;
  p.num_bags = static_cast<uint64_t>(hp->num_tables) * hp->batch;
  p.N = hp->num_indices;
  p.M = static_cast<uint32_t>(M);
  p.a = hp->a;
  p.b = hp->b;
  p.T = hp->num_tables;
  p.B = hp->batch;
  p.C = static_cast<uint32_t>(d / Z);
  p.Z = static_cast<uint32_t>(Z);
  p.d = static_cast<uint32_t>(d);
  p.TC = p.T * p.C;
  p.row_stride = p.T * p.d;
  p.sign_mode = (hp->flags & PSS_SIGN_MASK) >> 2;
  p.s_alpha = p.s_beta = p.a2 = 0;
  if (p.sign_mode) {
    // h2_0 = a2 * key_0 + b2 = alpha * h_0 + beta (mod p), key_0 = (h_0 - b) / a
    const uint32_t a_inv = pss::pow_mod_p(p.a, PSS_PRIME - 2);
    p.a2 = hp->sign_a;
    p.s_alpha = pss::mod_p(static_cast<uint64_t>(hp->sign_a) * a_inv);
    const uint32_t ab = pss::mod_p(static_cast<uint64_t>(p.s_alpha) * p.b);
    p.s_beta = pss::mod_p(static_cast<uint64_t>(hp->sign_b) + PSS_PRIME - ab);
  }
  p.mean = (hp->flags & PSS_POOL_MEAN) ? 1u : 0u;
  p.idx32 = (hp->flags & PSS_INDEX_I32) ? 1u : 0u;
  p.rows_bf16 = (hp->flags & PSS_ROWS_BF16) ? 1u : 0u;
  return p;
}

// One memory pool per device, created on first use, that keeps what it has
// reserved (release threshold = max) so steady-state calls do not go back to
// the driver for scratch space.
std::mutex g_pool_mu;
std::map<int, hipMemPool_t> g_pools;

// Upper bound on the unique locations of a batch: every lookup reads d
// elements, and there are M elements.
int64_t sparse_capacity(int64_t M, const KParams& p) {
  const int64_t nd = p.N * static_cast<int64_t>(p.d);
  return nd < M ? nd : M;
}

// AUTO's choice (paper Sec. 3: dense gradients win at high compression,
// sparse ones cost the same at any compression).  A fused SGD update costs
// nothing per element of M, so SORTED.  An unfused update (Adagrad, bf16
// storage) pays a pass over all M elements; when M exceeds 16 times the
// batch's N*d reads (low compression) the sparse path, whose cost follows
// the batch, is cheaper: measured crossover between 10x and 100x compression
// at batch 10240, d = 128.
uint32_t auto_variant(int64_t M, const KParams& p, bool unfused, bool sparse_fits) {
  const int64_t reads = p.N * static_cast<int64_t>(p.d);
  if (unfused && sparse_fits && M > 16 * reads) return PSS_BWD_SPARSE;
  return PSS_BWD_SORTED;
}

// AUTO's deposit order for the SORTED variant: by address when a chunk has
// at most 2 elements and the array lies beyond the memory-side cache
// (M * 4 > 256 MiB, where tables are large and lookups seldom repeat).
// The address sort costs the same for every Z (it moves N * d records);
// grouping by token leaves one atomic per lookup and chunk when tokens do
// not repeat.  Measured on a 26-table one-hot batch of uniform indices
// (4 GB array): Z = 1 12.8 -> 5.7 ms, Z = 2 6.7 -> 5.6 ms by address, but
// Z = 4 3.7 against 5.4 ms and Z = 8 2.2 against 5.3 ms by token.  Skewed
// tokens make the grouping cheaper still, hence the array-size condition.
// Needs N * d < 2^31 records.
constexpr uint32_t kAddrMaxZ = 2;
bool by_address_auto(int64_t M, const KParams& p) {
  return p.Z <= kAddrMaxZ && M * static_cast<int64_t>(sizeof(float)) > (256ll << 20) &&
         p.N * static_cast<int64_t>(p.d) < (1ll << 31);
}

// Chunks of at least this many elements deposit by address as run sums
// (grouped by token first): a run's chunk is then a read of whole lines.
constexpr uint32_t kRunsMinZ = 64;
bool runs_fit(const KParams& p) {
  return p.Z >= kRunsMinZ && p.N * static_cast<int64_t>(p.C) < (1ll << 31) &&
         p.N * static_cast<int64_t>(p.d) < (1ll << 31);
}
// AUTO never picks them: with chunks that long the atomics move whole lines
// at the memory system's streaming rate, and writing the run sums out and
// reading them back costs as much (row-hash workload: backward 1.66 ms
// against 1.11-1.23 ms).  Asked for with the flag they give the same update
// with every sum taken in a fixed order: the result does not change from
// run to run.

hipError_t pool_for_current_device(hipMemPool_t* out) {
  int dev = 0;
  hipError_t st = hipGetDevice(&dev);
  if (st != hipSuccess) return st;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  auto it = g_pools.find(dev);
  if (it != g_pools.end()) {
    *out = it->second;
    return hipSuccess;
  }
  hipMemPoolProps props;
  memset(&props, 0, sizeof(props));
  props.allocType = hipMemAllocationTypePinned;
  props.handleTypes = hipMemHandleTypeNone;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = dev;
  hipMemPool_t pool = nullptr;
  st = hipMemPoolCreate(&pool, &props);
  if (st != hipSuccess) return st;
  uint64_t threshold = UINT64_MAX;
  st = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &threshold);
  if (st != hipSuccess) {
    (void)hipMemPoolDestroy(pool);
    return st;
  }
  g_pools[dev] = pool;
  *out = pool;
  return hipSuccess;
}

int scratch_alloc(void** ptr, size_t bytes, hipStream_t stream) {
  hipMemPool_t pool = nullptr;
  if (pool_for_current_device(&pool) != hipSuccess) return PSS_ERR_HIP;
  const hipError_t st = hipMallocFromPoolAsync(ptr, bytes, pool, stream);
  if (st == hipErrorOutOfMemory) return PSS_ERR_NO_MEMORY;
  return st == hipSuccess ? PSS_OK : PSS_ERR_HIP;
}

// Scratch kept between calls, one buffer per (device, stream), as large as
// the largest call on that stream so far.  A pool allocation and its
// stream-ordered free per call cost the stream a marker between steps and
// block the host until earlier frees have completed; a kept buffer costs
// neither.  Work on one stream runs in order, so consecutive calls on it
// may share the buffer; a call holds the buffer's lock from taking it until
// its work is enqueued, so that calls made on one stream from several host
// threads do not interleave their kernels.  Streams are told apart by
// handle: the runtime keeps a stream object (whose address is the handle)
// alive while commands enqueued on it are pending, so a handle is reused
// only after the work of the stream it named has finished.
struct KeptScratch {
  std::mutex mu;
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_kept_mu;  // guards the map (std::map nodes do not move)
std::map<std::pair<int, uintptr_t>, KeptScratch> g_kept;

// Scratch of one call for work enqueued on `stream`: a kept buffer, or a
// pool allocation returned on the stream by done() (while the stream is
// being captured into a graph, which then owns its allocation and whose
// replays on other streams must not share a kept buffer, or when the
// capture status cannot be read).
class CallScratch {
 public:
  int take(size_t bytes, hipStream_t stream) {
    stream_ = stream;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    int dev = 0;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone ||
        hipGetDevice(&dev) != hipSuccess) {
      (void)hipGetLastError();
      const int st = scratch_alloc(&ptr_, bytes, stream);
      if (st != PSS_OK) ptr_ = nullptr;
      return st;
    }
    {
      std::lock_guard<std::mutex> map_lock(g_kept_mu);
      kept_ = &g_kept[{dev, reinterpret_cast<uintptr_t>(stream)}];
    }
    lock_ = std::unique_lock<std::mutex>(kept_->mu);
    if (kept_->bytes < bytes) {
      // the smaller buffer goes back to the pool after the work already
      // enqueued on the stream
      if (kept_->ptr != nullptr && hipFreeAsync(kept_->ptr, stream) != hipSuccess) return PSS_ERR_HIP;
      kept_->ptr = nullptr;
      kept_->bytes = 0;
      const int st = scratch_alloc(&kept_->ptr, bytes, stream);
      if (st != PSS_OK) {
        kept_->ptr = nullptr;
        return st;
      }
      kept_->bytes = bytes;
    }
    ptr_ = kept_->ptr;
    return PSS_OK;
  }
  void* ptr() const { return ptr_; }
  // Call once the work using the scratch is enqueued.
  hipError_t done() {
    hipError_t e = hipSuccess;
    if (kept_ == nullptr && ptr_ != nullptr) e = hipFreeAsync(ptr_, stream_);
    ptr_ = nullptr;
    if (lock_.owns_lock()) lock_.unlock();
    return e;
  }
  ~CallScratch() { (void)done(); }

 private:
  hipStream_t stream_ = nullptr;
  void* ptr_ = nullptr;
  KeptScratch* kept_ = nullptr;
  std::unique_lock<std::mutex> lock_;
};

// Grouping prepared by a forward call with PSS_PREPARE_BACKWARD, one slot
// per (device, caller stream).  The grouping runs on a library stream of its
// own, after the caller's stream has reached the forward call (event
// `start`), so it overlaps the forward kernel; `ready` marks its end.  The
// next backward on the caller's stream with the same indices, offsets and
// grouping parameters waits for `ready` and reuses the pairs instead of
// grouping again.  A later prepare on the same stream reuses the buffer: its
// grouping waits for `start`, recorded after every earlier call on the
// caller's stream (including the backward that read the buffer).
//
// A forward that runs the streamed kernel writes the grouping's first stage
// (keygen) itself instead (`fused`): it reads the batch's index and offset
// entries anyway.  Everything then happens on the caller's stream (no side
// stream, no events), and the backward finishes the grouping (the radix
// pass) before its reduction.
struct Prepared {
  std::mutex mu;
  hipStream_t side = nullptr;
  hipEvent_t start = nullptr;
  hipEvent_t ready = nullptr;
  void* buf = nullptr;
  size_t bytes = 0;
  bool valid = false;  // a grouping waits for its backward
  bool fused = false;  // valid: its keygen stage was written by the forward kernel
  const void* indices = nullptr;
  const void* offsets = nullptr;
  KParams made{};
  pss::GroupedPairs pairs;
};
std::mutex g_prep_mu;  // guards the map (std::map nodes do not move)
std::map<std::pair<int, uintptr_t>, Prepared> g_prep;

// Parameters the grouping depends on.
bool same_grouping(const KParams& x, const KParams& y) {
  return x.N == y.N && x.num_bags == y.num_bags && x.T == y.T && x.B == y.B && x.C == y.C &&
         x.a == y.a && x.b == y.b && x.mean == y.mean && x.idx32 == y.idx32;
}

bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return true;  // unknown: treat as captured (no side stream)
  }
  return cs != hipStreamCaptureStatusNone;
}

int prepare_backward(const KParams& p, const void* indices, const void* offsets,
                     hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return PSS_ERR_HIP;
  Prepared* pr = nullptr;
  {
    std::lock_guard<std::mutex> map_lock(g_prep_mu);
    pr = &g_prep[{dev, reinterpret_cast<uintptr_t>(stream)}];
  }
  std::lock_guard<std::mutex> lock(pr->mu);
  // A grouping that no backward used is dropped; the caller's stream first
  // waits for it, so that work the caller orders after this call (freeing or
  // refilling the old batch's indices) also follows the old grouping's reads.
  if (pr->valid && !pr->fused && hipStreamWaitEvent(stream, pr->ready, 0) != hipSuccess) {
    pr->valid = false;
    return PSS_ERR_HIP;
  }
  pr->valid = false;
  pr->fused = false;
  // created on first use (each one again if an earlier creation failed);
  // both events order work on this device only, so they release at device
  // scope (a system-scope release would write back the L2s for the host)
  if (pr->side == nullptr && hipStreamCreateWithFlags(&pr->side, hipStreamNonBlocking) != hipSuccess) {
    pr->side = nullptr;
    return PSS_ERR_HIP;
  }
  for (hipEvent_t* ev : {&pr->start, &pr->ready}) {
    if (*ev == nullptr &&
        hipEventCreateWithFlags(ev, hipEventDisableTiming | hipEventReleaseToDevice) != hipSuccess) {
      *ev = nullptr;
      return PSS_ERR_HIP;
    }
  }
  if (hipEventRecord(pr->start, stream) != hipSuccess ||
      hipStreamWaitEvent(pr->side, pr->start, 0) != hipSuccess)
    return PSS_ERR_HIP;
  const size_t need = pss::sorted_workspace_bytes(p);
  if (pr->bytes < need) {
    // both stream-ordered on the library stream, after the caller's earlier work
    if (pr->buf != nullptr && hipFreeAsync(pr->buf, pr->side) != hipSuccess) return PSS_ERR_HIP;
    pr->buf = nullptr;
    pr->bytes = 0;
    const int st = scratch_alloc(&pr->buf, need, pr->side);
    if (st != PSS_OK) {
      pr->buf = nullptr;
      return st;
    }
    pr->bytes = need;
  }
  if (pss::launch_group_sorted(p, indices, offsets, pr->buf, pr->side, &pr->pairs) != hipSuccess ||
      hipEventRecord(pr->ready, pr->side) != hipSuccess)
    return PSS_ERR_HIP;
  pr->indices = indices;
  pr->offsets = offsets;
  pr->made = p;
  pr->valid = true;
  return PSS_OK;
}

// Sets up the slot for a grouping whose keygen stage the streamed forward
// kernel writes on the caller's stream (the buffer is allocated, and an
// unused earlier grouping dropped, in stream order); *kg gets the stage's
// layout in the slot's buffer.  The slot becomes valid only through
// mark_fused, once the forward kernel has been enqueued.
int prepare_fused(const KParams& p, const void* indices, const void* offsets, hipStream_t stream,
                  pss::KeygenOut* kg, Prepared** slot) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return PSS_ERR_HIP;
  Prepared* pr = nullptr;
  {
    std::lock_guard<std::mutex> map_lock(g_prep_mu);
    pr = &g_prep[{dev, reinterpret_cast<uintptr_t>(stream)}];
  }
  std::lock_guard<std::mutex> lock(pr->mu);
  // an unused grouping made on the library stream may still be reading its
  // batch or writing the buffer: the caller's stream waits for it
  if (pr->valid && !pr->fused && hipStreamWaitEvent(stream, pr->ready, 0) != hipSuccess) {
    pr->valid = false;
    return PSS_ERR_HIP;
  }
  pr->valid = false;
  pr->fused = false;
  const size_t need = pss::sorted_workspace_bytes(p);
  if (pr->bytes < need) {
    if (pr->buf != nullptr && hipFreeAsync(pr->buf, stream) != hipSuccess) return PSS_ERR_HIP;
    pr->buf = nullptr;
    pr->bytes = 0;
    const int st = scratch_alloc(&pr->buf, need, stream);
    if (st != PSS_OK) {
      pr->buf = nullptr;
      return st;
    }
    pr->bytes = need;
  }
  *kg = pss::keygen_layout(p, pr->buf);
  pr->indices = indices;
  pr->offsets = offsets;
  pr->made = p;
  *slot = pr;
  return PSS_OK;
}

void mark_fused(Prepared* pr) {
  std::lock_guard<std::mutex> lock(pr->mu);
  pr->valid = true;
  pr->fused = true;
}

// The grouped pairs of a prepared grouping, on `stream`: wait for the
// library stream's grouping, or finish the one whose keygen stage the
// forward wrote.
hipError_t prepared_pairs(Prepared* prep, const KParams& p, hipStream_t stream,
                          pss::GroupedPairs* pairs) {
  if (prep->fused) return pss::finish_group_sorted(p, prep->buf, true, stream, pairs);
  *pairs = prep->pairs;
  return hipStreamWaitEvent(stream, prep->ready, 0);
}

// The grouping prepared by the last forward on `stream`, if it was made for
// this batch and `usable`; nullptr otherwise.  A prepared grouping serves the
// next backward call on its stream only: this call drops it either way.  On
// success *lock holds the slot until the caller's work is enqueued.
Prepared* take_prepared(hipStream_t stream, const void* indices, const void* offsets,
                        const KParams& p, bool usable, std::unique_lock<std::mutex>* lock) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  Prepared* pr = nullptr;
  {
    std::lock_guard<std::mutex> map_lock(g_prep_mu);
    auto it = g_prep.find({dev, reinterpret_cast<uintptr_t>(stream)});
    if (it == g_prep.end()) return nullptr;
    pr = &it->second;
  }
  std::unique_lock<std::mutex> slot(pr->mu);
  const bool match = pr->valid && pr->indices == indices && pr->offsets == offsets &&
                     same_grouping(pr->made, p);
  if (pr->valid && !pr->fused && (!match || !usable)) {
    // dropped unused: the caller's stream waits for the grouping (it may
    // still be reading its batch's indices and offsets)
    if (hipStreamWaitEvent(stream, pr->ready, 0) != hipSuccess) (void)hipGetLastError();
  }
  pr->valid = false;
  if (!match || !usable) return nullptr;
  *lock = std::move(slot);
  return pr;
}

int hip_status(hipError_t st) { return st == hipSuccess ? PSS_OK : PSS_ERR_HIP; }

// Whether a backward with these flags can run the SORTED variant grouped by
// token (the grouping that pss_prepare_backward makes ahead): AUTO or SORTED,
// not sorted by address (asked for, or AUTO's choice for the shape).
bool groups_by_token(int64_t M, const KParams& p, const pss_hash_params* hp) {
  const uint32_t variant = hp->flags & PSS_BWD_MASK;
  if (variant != PSS_BWD_AUTO && variant != PSS_BWD_SORTED) return false;
  // by address: grouped only as run sums (chunks of 64 elements or more)
  if (hp->flags & PSS_DEPOSIT_BY_ADDRESS) return p.Z >= kRunsMinZ;
  return !(variant == PSS_BWD_AUTO && by_address_auto(M, p));
}

// One backward call: the variant that runs and the scratch it needs.
struct BackwardPlan {
  KParams p;
  uint32_t variant = PSS_BWD_SORTED;  // ATOMIC, SORTED or SPARSE
  bool by_address = false;            // SORTED: records sorted by address tile
  bool runs = false;                  // ... the records being run sums (grouped by token)
  bool bf16 = false;
  bool fused = false;   // SGD on float32 storage: deposits go into `shared`
  size_t g_bytes = 0;   // float32 gradient buffer (unfused updates), 256-aligned
  size_t runs_bytes = 0;  // run sums by address: records and payload, after G
  size_t ws_bytes = 0;  // grouping (SORTED) or sparse workspace, after those
};
constexpr int kNothingToDo = -1;  // no lookups: G == 0, nothing changes

// Argument checks of the backward entry points (host only, before anything
// is enqueued) and the plan.  Returns PSS_OK, kNothingToDo or an error.
int plan_backward(void* shared, float* state, int64_t M, int32_t Z, int32_t d,
                  const pss_hash_params* hp, const void* indices, const void* offsets,
                  const void* grad_out, float lr, BackwardPlan* plan) {
  const int st = check_common(M, Z, d, hp);
  if (st != PSS_OK) return st;
  if (shared == nullptr || offsets == nullptr || grad_out == nullptr) return PSS_ERR_INVALID_ARG;
  if (indices == nullptr && hp->num_indices > 0) return PSS_ERR_INVALID_ARG;
  if (!isfinite(lr)) return PSS_ERR_INVALID_ARG;
  if (state != nullptr && !(hp->eps >= 0.f && isfinite(hp->eps))) return PSS_ERR_INVALID_ARG;
  plan->p = make_params(M, Z, d, hp);
  const KParams& p = plan->p;
  plan->bf16 = hp->weight_dtype == PSS_BF16;
  const bool sparse_fits = p.N * static_cast<int64_t>(p.C) < (1ll << 31);
  uint32_t variant = hp->flags & PSS_BWD_MASK;
  const bool addr_asked = (hp->flags & PSS_DEPOSIT_BY_ADDRESS) != 0;
  if (variant == PSS_BWD_SPARSE && !sparse_fits) return PSS_ERR_UNSUPPORTED;
  if (addr_asked && (variant == PSS_BWD_ATOMIC || variant == PSS_BWD_SPARSE))
    return PSS_ERR_UNSUPPORTED;
  if (addr_asked && p.N * static_cast<int64_t>(p.d) >= (1ll << 31)) return PSS_ERR_UNSUPPORTED;
  if (addr_asked && p.Z >= kRunsMinZ && !runs_fit(p)) return PSS_ERR_UNSUPPORTED;
  if (p.N == 0) return kNothingToDo;
  const bool auto_pick = variant == PSS_BWD_AUTO;
  if (auto_pick) variant = auto_variant(M, p, state != nullptr || plan->bf16, sparse_fits);
  plan->variant = variant;
  plan->by_address = variant == PSS_BWD_SORTED && (addr_asked || (auto_pick && by_address_auto(M, p)));
  plan->runs = plan->by_address && p.Z >= kRunsMinZ;
  if (variant == PSS_BWD_SPARSE) {
    // Alg. 1 sparse branch: 256 bytes for the unique count, then its workspace
    plan->ws_bytes = 256 + pss::sparse_workspace_bytes(p);
    return PSS_OK;
  }
  // SGD on float32 storage is linear in G: deposit -lr * grad directly into
  // the shared array.  Otherwise deposit G into a scratch buffer first.
  plan->fused = state == nullptr && !plan->bf16;
  if (plan->runs) {
    // the tiles update `shared` (and `state`) directly: no G buffer
    plan->runs_bytes = (pss::runs_workspace_bytes(p) + 255) & ~size_t(255);
    plan->ws_bytes = pss::sorted_workspace_bytes(p);
    return PSS_OK;
  }
  plan->g_bytes = plan->fused ? 0 : (static_cast<size_t>(M) * sizeof(float) + 255) & ~size_t(255);
  plan->ws_bytes = variant != PSS_BWD_SORTED ? 0
                   : plan->by_address       ? pss::addr_workspace_bytes(p)
                                            : pss::sorted_workspace_bytes(p);
  return PSS_OK;
}

// Enqueues the planned backward on `stream`.  ws: scratch of at least
// plan.g_bytes + plan.runs_bytes + plan.ws_bytes bytes; prep: a grouping made ahead for this
// batch (SORTED only), or null.
hipError_t enqueue_backward(const BackwardPlan& plan, void* shared, float* state, float eps,
                            const void* indices, const void* offsets, const void* grad_out,
                            float lr, void* ws, Prepared* prep, hipStream_t stream) {
  const KParams& p = plan.p;
  if (plan.variant == PSS_BWD_SPARSE) {
    // the optimizer is applied at each unique location as it is summed
    uint32_t* count = static_cast<uint32_t*>(ws);
    return pss::launch_sparse_update(p, indices, offsets, grad_out, static_cast<char*>(ws) + 256,
                                     count, shared, plan.bf16, state, lr, eps, stream);
  }
  if (plan.runs) {
    void* runs_ws = static_cast<char*>(ws) + plan.g_bytes;
    void* group_ws = static_cast<char*>(runs_ws) + plan.runs_bytes;
    pss::GroupedPairs pairs;
    hipError_t e = hipSuccess;
    if (prep != nullptr) {
      // the grouping made ahead (on the library stream, or begun by the
      // forward kernel)
      e = prepared_pairs(prep, p, stream, &pairs);
    } else {
      e = pss::launch_group_sorted(p, indices, offsets, group_ws, stream, &pairs);
    }
    if (e == hipSuccess)
      e = pss::launch_deposit_runs(shared, plan.bf16, state, lr, eps, p, pairs, grad_out, runs_ws,
                                   stream);
    return e;
  }
  float* dst = plan.fused ? static_cast<float*>(shared) : static_cast<float*>(ws);
  void* sort_ws = static_cast<char*>(ws) + plan.g_bytes;
  const float scale = plan.fused ? -lr : 1.f;
  const int64_t M = p.M;
  hipError_t e = hipSuccess;
  if (plan.by_address) {
    // every tile of G is stored whole: no zero-fill
    e = pss::launch_deposit_addr(dst, !plan.fused, scale, p, indices, offsets, grad_out, sort_ws,
                                 stream);
    if (e == hipSuccess && !plan.fused)
      e = pss::launch_optimizer(shared, plan.bf16, state, dst, M, lr, eps, stream);
    return e;
  }
  if (!plan.fused) e = pss::launch_zero(dst, M, stream);
  if (e == hipSuccess && prep != nullptr) {
    // the grouping made ahead (on the library stream, or begun by the
    // forward kernel)
    pss::GroupedPairs pairs;
    e = prepared_pairs(prep, p, stream, &pairs);
    if (e == hipSuccess) e = pss::launch_reduce_sorted(dst, scale, p, pairs, grad_out, stream);
  } else if (e == hipSuccess) {
    e = plan.variant == PSS_BWD_SORTED
            ? pss::launch_deposit_sorted(dst, scale, p, indices, offsets, grad_out, sort_ws, stream)
            : pss::launch_deposit_atomic(dst, scale, p, indices, offsets, grad_out, stream);
  }
  if (e == hipSuccess && !plan.fused)
    e = pss::launch_optimizer(shared, plan.bf16, state, dst, M, lr, eps, stream);
  return e;
}

// ---------------------------------------------------------------------------
// Scratch of pss_backward_update_noalloc: a static device array (each GPU
// holds its own copy, from the library's first use on it until the process
// ends).  In host code `scratch` names a host-side stand-in, not the device
// memory: its device address is taken once per device with
// hipGetSymbolAddress, with that device current, and only that address is
// passed to kernels.
// ---------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = static_cast<size_t>(PSS_NOALLOC_SCRATCH_BYTES);
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_static_mu;
std::map<int, void*> g_static_ptr;  // device -> device address of `scratch`

hipError_t static_scratch_for_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_static_mu);
  auto it = g_static_ptr.find(dev);
  if (it != g_static_ptr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || ptr == nullptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
  g_static_ptr[dev] = ptr;
  *out = ptr;
  return hipSuccess;
}

uint64_t splitmix64_next(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace

extern "C" {

int pss_hash_params_from_seed(uint64_t seed, pss_hash_params* p) {
  if (p == nullptr) return PSS_ERR_INVALID_ARG;
  uint64_t state = seed;
  const uint64_t x1 = splitmix64_next(&state);
  const uint64_t x2 = splitmix64_next(&state);
  const uint64_t x3 = splitmix64_next(&state);
  const uint64_t x4 = splitmix64_next(&state);
  p->a = static_cast<uint32_t>(1 + x1 % (PSS_PRIME - 1));
  p->b = static_cast<uint32_t>(x2 % PSS_PRIME);
  p->sign_a = static_cast<uint32_t>(1 + x3 % (PSS_PRIME - 1));
  p->sign_b = static_cast<uint32_t>(x4 % PSS_PRIME);
  return PSS_OK;
}

int pss_forward(const void* shared, int64_t M, int32_t Z, int32_t d,
                const pss_hash_params* hash_params, const void* indices,
                const void* offsets, void* out, hipStream_t stream) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  if (shared == nullptr || offsets == nullptr || out == nullptr) return PSS_ERR_INVALID_ARG;
  if (indices == nullptr && hash_params->num_indices > 0) return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  // The grouping is only reused by the SORTED backward grouped by token
  // (AUTO's usual choice when the update is fused), and only outside graph
  // capture.  The preparation only saves the backward some work: if it cannot be set
  // up (no memory for its buffer, a failed runtime call), the forward runs
  // anyway and the backward groups the batch itself.
  const bool bf16 = hash_params->weight_dtype == PSS_BF16;
  pss::KeygenOut kg;
  Prepared* fused = nullptr;
  if ((hash_params->flags & PSS_PREPARE_BACKWARD) && p.N > 0 && groups_by_token(M, p, hash_params) &&
      !capturing(stream)) {
    // the streamed kernel writes the grouping's keygen stage itself; other
    // forwards leave the grouping to the library stream
    if (pss::forward_streams(p, bf16)) {
      if (prepare_fused(p, indices, offsets, stream, &kg, &fused) != PSS_OK) {
        (void)hipGetLastError();
        fused = nullptr;
      }
    } else if (prepare_backward(p, indices, offsets, stream) != PSS_OK) {
      (void)hipGetLastError();
    }
  }
  const hipError_t e = pss::launch_forward(shared, bf16, p, indices, offsets, out, stream,
                                           fused != nullptr ? &kg : nullptr);
  if (e == hipSuccess && fused != nullptr) mark_fused(fused);
  return hip_status(e);
}

int pss_prepare_backward(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                         const void* indices, const void* offsets, hipStream_t stream) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  if (offsets == nullptr) return PSS_ERR_INVALID_ARG;
  if (indices == nullptr && hash_params->num_indices > 0) return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  if (p.N == 0 || !groups_by_token(M, p, hash_params) || capturing(stream)) return PSS_OK;
  const int ps = prepare_backward(p, indices, offsets, stream);
  if (ps != PSS_OK) (void)hipGetLastError();
  return ps;
}

int pss_backward_update(void* shared, float* state, int64_t M, int32_t Z, int32_t d,
                        const pss_hash_params* hash_params, const void* indices,
                        const void* offsets, const void* grad_out, float lr,
                        hipStream_t stream) {
  BackwardPlan plan;
  const int st = plan_backward(shared, state, M, Z, d, hash_params, indices, offsets, grad_out, lr,
                               &plan);
  if (st != PSS_OK) return st == kNothingToDo ? PSS_OK : st;
  std::unique_lock<std::mutex> prep_lock;
  Prepared* prep = take_prepared(stream, indices, offsets, plan.p,
                                 plan.variant == PSS_BWD_SORTED &&
                                     (!plan.by_address || plan.runs) && !capturing(stream),
                                 &prep_lock);
  if (prep != nullptr) plan.ws_bytes = 0;  // the grouping is already made
  CallScratch scratch;
  const size_t need = plan.g_bytes + plan.runs_bytes + plan.ws_bytes;
  if (need > 0) {
    const int ts = scratch.take(need, stream);
    if (ts != PSS_OK) return ts;
  }
  const hipError_t e = enqueue_backward(plan, shared, state, hash_params->eps, indices, offsets,
                                        grad_out, lr, scratch.ptr(), prep, stream);
  const hipError_t ef = scratch.done();
  return (e != hipSuccess || ef != hipSuccess) ? PSS_ERR_HIP : PSS_OK;
}

int pss_backward_update_noalloc(void* shared, float* state, int64_t M, int32_t Z, int32_t d,
                                const pss_hash_params* hash_params, const void* indices,
                                const void* offsets, const void* grad_out, float lr,
                                hipStream_t stream) {
  BackwardPlan plan;
  const int st = plan_backward(shared, state, M, Z, d, hash_params, indices, offsets, grad_out, lr,
                               &plan);
  if (st != PSS_OK) return st == kNothingToDo ? PSS_OK : st;
  const size_t need = plan.g_bytes + plan.runs_bytes + plan.ws_bytes;
  if (need > kStaticScratchBytes) return PSS_ERR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if (need > 0 && static_scratch_for_current_device(&ws) != hipSuccess)
    return PSS_ERR_HIP;
  return enqueue_backward(plan, shared, state, hash_params->eps, indices, offsets, grad_out, lr, ws,
                          nullptr, stream) == hipSuccess
             ? PSS_OK
             : PSS_ERR_HIP;
}

int pss_gradient_sparse(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const void* indices, const void* offsets, const void* grad_out,
                        uint32_t* locations, float* values, int64_t capacity, int64_t* num_unique,
                        hipStream_t stream) {
  int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  if (offsets == nullptr || grad_out == nullptr || num_unique == nullptr) return PSS_ERR_INVALID_ARG;
  if (indices == nullptr && hash_params->num_indices > 0) return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  if (p.N * static_cast<int64_t>(p.C) >= (1ll << 31)) return PSS_ERR_UNSUPPORTED;
  if (capacity < sparse_capacity(M, p)) return PSS_ERR_INVALID_ARG;
  if (p.N > 0 && (locations == nullptr || values == nullptr)) return PSS_ERR_INVALID_ARG;
  const size_t ws_bytes = 256 + (p.N > 0 ? pss::sparse_workspace_bytes(p) : 0);
  CallScratch scratch;
  st = scratch.take(ws_bytes, stream);
  if (st != PSS_OK) return st;
  void* ws = scratch.ptr();
  uint32_t* count = static_cast<uint32_t*>(ws);
  hipError_t e = hipSuccess;
  if (p.N == 0) {
    e = pss::launch_zero(reinterpret_cast<float*>(count), 1, stream);
  } else {
    e = pss::launch_gradient_sparse(p, indices, offsets, grad_out, static_cast<char*>(ws) + 256,
                                    locations, values, capacity, count, stream);
  }
  if (e == hipSuccess) e = pss::launch_store_count(count, num_unique, stream);
  const hipError_t ef = scratch.done();
  return (e != hipSuccess || ef != hipSuccess) ? PSS_ERR_HIP : PSS_OK;
}

int pss_debug_addresses(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const void* indices, const void* offsets, uint32_t* base_out,
                        hipStream_t stream) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  if (offsets == nullptr) return PSS_ERR_INVALID_ARG;
  if (hash_params->num_indices > 0 && (indices == nullptr || base_out == nullptr))
    return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  return hip_status(pss::launch_debug_addresses(p, indices, offsets, base_out, nullptr, stream));
}

int pss_debug_signs(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                    const void* indices, const void* offsets, int8_t* sign_out,
                    hipStream_t stream) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  if (offsets == nullptr) return PSS_ERR_INVALID_ARG;
  if (hash_params->num_indices > 0 && (indices == nullptr || sign_out == nullptr))
    return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  return hip_status(pss::launch_debug_addresses(p, indices, offsets, nullptr, sign_out, stream));
}

int pss_debug_reduce_events(void* before, void* after) {
  if ((before == nullptr) != (after == nullptr)) return PSS_ERR_INVALID_ARG;
  pss::set_reduce_events(static_cast<hipEvent_t>(before), static_cast<hipEvent_t>(after));
  return PSS_OK;
}

int pss_release_scratch(void) {
  std::lock_guard<std::mutex> lock(g_kept_mu);
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return PSS_ERR_HIP;
  int status = PSS_OK;
  for (auto& kv : g_kept) {
    std::lock_guard<std::mutex> entry_lock(kv.second.mu);
    if (kv.second.ptr == nullptr) continue;
    // the buffer may still be in use by work enqueued on its stream
    if (hipSetDevice(kv.first.first) != hipSuccess || hipDeviceSynchronize() != hipSuccess ||
        hipFreeAsync(kv.second.ptr, nullptr) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
      status = PSS_ERR_HIP;
  }
  g_kept.clear();
  {
    std::lock_guard<std::mutex> map_lock(g_prep_mu);
    for (auto& kv : g_prep) {
      Prepared& pr = kv.second;
      std::lock_guard<std::mutex> entry_lock(pr.mu);
      if (hipSetDevice(kv.first.first) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
        status = PSS_ERR_HIP;
      if (pr.buf != nullptr && (hipFreeAsync(pr.buf, nullptr) != hipSuccess ||
                                hipDeviceSynchronize() != hipSuccess))
        status = PSS_ERR_HIP;
      if (pr.start != nullptr && hipEventDestroy(pr.start) != hipSuccess) status = PSS_ERR_HIP;
      if (pr.ready != nullptr && hipEventDestroy(pr.ready) != hipSuccess) status = PSS_ERR_HIP;
      if (pr.side != nullptr && hipStreamDestroy(pr.side) != hipSuccess) status = PSS_ERR_HIP;
    }
    g_prep.clear();
  }
  {
    // the pools last: every buffer taken from them has been returned above
    std::lock_guard<std::mutex> pool_lock(g_pool_mu);
    for (auto& kv : g_pools) {
      if (hipSetDevice(kv.first) != hipSuccess || hipDeviceSynchronize() != hipSuccess ||
          hipMemPoolDestroy(kv.second) != hipSuccess)
        status = PSS_ERR_HIP;
    }
    g_pools.clear();
  }
  if (hipSetDevice(cur) != hipSuccess) status = PSS_ERR_HIP;
  return status;
}

int pss_validate_offsets_host(const int64_t* offsets, int64_t num_bags, int64_t N) {
  if (offsets == nullptr || num_bags < 0 || N < 0) return PSS_ERR_INVALID_ARG;
  if (offsets[0] != 0 || offsets[num_bags] != N) return PSS_ERR_INVALID_ARG;
  for (int64_t g = 0; g < num_bags; ++g)
    if (offsets[g + 1] < offsets[g]) return PSS_ERR_INVALID_ARG;
  return PSS_OK;
}

int pss_hash_bases_host(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const int64_t* indices, const int64_t* offsets, uint32_t* base_out) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  const int64_t bags = static_cast<int64_t>(hash_params->num_tables) * hash_params->batch;
  const int64_t N = hash_params->num_indices;
  if (pss_validate_offsets_host(offsets, bags, N) != PSS_OK) return PSS_ERR_INVALID_ARG;
  if (N > 0 && (indices == nullptr || base_out == nullptr)) return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  for (int64_t g = 0; g < bags; ++g) {
    const uint32_t t = static_cast<uint32_t>(g / p.B);
    for (int64_t e = offsets[g]; e < offsets[g + 1]; ++e) {
      const uint32_t i = static_cast<uint32_t>(indices[e]);
      for (uint32_t j = 0; j < p.C; ++j)
        base_out[e * p.C + j] = pss::chunk_base(i, t, j, p.C, p.TC, p.a, p.b, p.fm_c, p.M);
    }
  }
  return PSS_OK;
}

int pss_hash_signs_host(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const int64_t* indices, const int64_t* offsets, int8_t* sign_out) {
  const int st = check_common(M, Z, d, hash_params);
  if (st != PSS_OK) return st;
  const int64_t bags = static_cast<int64_t>(hash_params->num_tables) * hash_params->batch;
  const int64_t N = hash_params->num_indices;
  if (pss_validate_offsets_host(offsets, bags, N) != PSS_OK) return PSS_ERR_INVALID_ARG;
  if (N > 0 && (indices == nullptr || sign_out == nullptr)) return PSS_ERR_INVALID_ARG;
  const KParams p = make_params(M, Z, d, hash_params);
  for (int64_t g = 0; g < bags; ++g) {
    const uint32_t t = static_cast<uint32_t>(g / p.B);
    for (int64_t e = offsets[g]; e < offsets[g + 1]; ++e) {
      const uint32_t i = static_cast<uint32_t>(indices[e]);
      const uint32_t h0 = pss::item_hash(i, t * p.C, p.TC, p.a, p.b);
      const uint32_t h20 = p.sign_mode ? pss::sign_hash0(h0, p.s_alpha, p.s_beta) : 0u;
      for (uint32_t j = 0; j < p.C; ++j) {
        int8_t f = 1;
        if (p.sign_mode) {
          const uint32_t code =
              pss::sign_code(pss::add_mod_p(h20, pss::chunk_step(p.a2, j)), p.sign_mode);
          f = code == 0 ? 1 : (code == 1 ? -1 : 0);
        }
        sign_out[e * p.C + j] = f;
      }
    }
  }
  return PSS_OK;
}

const char* pss_status_string(int status) {
  switch (status) {
    case PSS_OK: return "ok";
    case PSS_ERR_INVALID_ARG: return "invalid argument";
    case PSS_ERR_UNSUPPORTED: return "unsupported argument combination";
    case PSS_ERR_HIP: return "HIP runtime or launch failure";
    case PSS_ERR_NO_MEMORY: return "out of device memory for scratch space";
    case PSS_ERR_SCRATCH_LIMIT:
      return "the call needs more scratch than the allocation-free entry point holds";
    default: return "unknown status";
  }
}

}  // extern "C"

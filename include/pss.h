/*
 * pss.h - C ABI of the hashed shared-memory embedding layer (PSS, ROBE-Z
 * mapping) for AMD Instinct MI355X (gfx950).
 *
 * The layer keeps ONE flat learnable array `shared` of M weights for all T
 * embedding tables.  Chunk j (dims [jZ, (j+1)Z)) of the embedding of token i
 * of table t is read from Z consecutive weights starting at a universal-hash
 * address (paper Sec. 2.5, "HashedNet and ROBE-Z"; universal hashing of the
 * mapping: Sec. 2.5, "Sparse JL with independence relaxation"):
 *
 *     C    = d / Z                          chunks per embedding
 *     key  = (i * T + t) * C + j            exact 64-bit integer
 *     h    = ((a * key + b) mod p) mod M    p = 2^31 - 1
 *     dim jZ + k of the embedding  =  shared[(h + k) mod M],  0 <= k < Z
 *
 * Forward (Sec. 2.4, forward(i) = (S e_i)^T M) sum-pools those embeddings
 * over each bag; backward (Sec. 2.4, backward(i, Delta) = (S e_i) Delta, and
 * Alg. 1) scatter-adds the output gradient onto the addresses that were read
 * and applies the optimizer step to `shared` in the same call.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Bags.  There are T*B bags, table-major: bag g = t*B + b holds the token
 *   indices indices[offsets[g] .. offsets[g+1]) of table t for sample b.
 *   offsets: int64[T*B + 1] (int32 with PSS_INDEX_I32), offsets[0] = 0,
 *   non-decreasing, offsets[T*B] = N.  indices: int64[N] (int32 with
 *   PSS_INDEX_I32), each in [0, 2^31).  Duplicate indices in a bag count
 *   twice; empty bags pool to zero.
 * Pooled rows.  out / grad_out are float32 [B][T*d] (bfloat16 bit patterns
 *   with PSS_ROWS_BF16), row-major: element (b, t*d + c) belongs to bag
 *   t*B + b, embedding dim c.
 * Options (pss_hash_params.flags, beside the backward variant):
 *   PSS_SIGN_PM1, PSS_SIGN_SPARSE  chunk signs (paper Sec. 2.5, sparse JL
 *     with independence relaxation: entries of S in {+1, -1, 0} drawn by a
 *     universal hash).  A second hash h2 = (sign_a * key + sign_b) mod p of
 *     the same key gives chunk (i, j) a factor s: PM1: s = -1 if
 *     h2 >= 2^30, else +1.  SPARSE: s = +1 if h2 < q, -1 if q <= h2 < 2q,
 *     else 0, with q = floor(p / 6).  The forward reads s * shared[...]; the
 *     backward deposits s * grad.  A chunk of factor 0 is not read: it adds
 *     nothing and receives nothing.
 *   PSS_POOL_MEAN  each bag's pooled row is divided by its number of items
 *     (torch.nn.EmbeddingBag mode "mean"); the backward deposits grad / |bag|.
 *   PSS_INDEX_I32  indices and offsets are int32.
 *   PSS_ROWS_BF16  out is written, and grad_out read, as bfloat16 (out is
 *     rounded to nearest even from the float32 result).
 *   PSS_DEPOSIT_BY_ADDRESS  with the SORTED variant (with AUTO: whenever
 *     AUTO picks SORTED): the deposit is ordered by address instead of made
 *     with float atomics to memory.
 *     The contributions are radix-sorted by address tile (2^14 elements)
 *     and each tile sums its contributions on chip and is updated once.
 *     - Z < 64: every (lookup, dim) contribution is its own (address, value)
 *       record; the tile is applied to the array (SGD on float32) or stored
 *       as that tile of the float32 gradient buffer before the optimizer
 *       pass.  16 B of scratch per (lookup, dim).  AUTO takes this by itself
 *       for chunks of at most 2 elements (Z <= 2) on an array beyond the
 *       memory-side cache (M * 4 > 256 MiB), where lookups seldom repeat
 *       and each contribution would otherwise be an atomic to its own line;
 *       from Z = 4 on, the grouped deposit's one atomic per chunk costs
 *       less than sorting every (lookup, dim) record.
 *     - Z >= 64: the lookups are grouped by token first (as SORTED does) and
 *       each run sum becomes one record per chunk (Z values); each tile adds
 *       the chunks reaching it in a fixed order and applies the optimizer to
 *       its elements in place (no gradient buffer, no dense pass).  Every
 *       sum is taken in a fixed order, so the update is bit-identical run to
 *       run.  Scratch: N * d floats of run sums plus 20 B per (lookup,
 *       chunk).  AUTO never takes this one (the atomic deposit of whole-line
 *       chunks is as fast); it uses a grouping made ahead by
 *       PSS_PREPARE_BACKWARD like SORTED.  Requires N * (d/Z) < 2^31.
 *     Both require N * d < 2^31 (else PSS_ERR_UNSUPPORTED); the flag is
 *     invalid with ATOMIC or SPARSE (PSS_ERR_UNSUPPORTED).
 *   PSS_PREPARE_BACKWARD  read by pss_forward only (the other calls ignore
 *     it; pss_prepare_backward does the same work as a call of its own): the
 *     forward also groups the batch's lookups by token for the backward.  A
 *     forward that runs its streamed kernel (one item per bag, d in {64,
 *     128, 256}, Z % 4 == 0, the shared array within 32 MiB) writes the
 *     grouping's first stage (every lookup's key and pooled row, and the
 *     first radix pass's digit counts) from that kernel, on `stream`, while
 *     it reads the batch's index and offset entries; the backward finishes
 *     the grouping on its stream.  Other forwards group the batch on a
 *     library-owned stream that runs beside the forward kernel.  The next
 *     pss_backward_update on the same stream uses that grouping when its
 *     indices and offsets pointers, batch shape, hash parameters and options
 *     match and it runs the SORTED variant grouped by token (AUTO's choice
 *     for SGD on float32 storage; also the run sums by address of
 *     PSS_DEPOSIT_BY_ADDRESS with Z >= 64); it drops the grouping either way.  The match is by pointer:
 *     the library records the indices and offsets pointers of the prepared
 *     batch (comparing them later, never reading through them after the
 *     grouping's own work) and cannot see their contents, so the caller must
 *     not change the contents of indices or offsets between the two calls (a
 *     backward on other contents at the same addresses would deposit at the
 *     prepared batch's addresses).  A forward without the flag leaves a
 *     prepared grouping in place, so that pss_prepare_backward, pss_forward
 *     and pss_backward_update may follow each other.  When a grouping is
 *     dropped unused (by a backward that does not match or cannot use it, or
 *     by a new preparation on the same stream), `stream` first waits for it:
 *     work the caller enqueues there afterwards follows its reads of the old
 *     indices and offsets.  Ignored while the stream is being captured into a
 *     graph, for an explicit ATOMIC or SPARSE variant and for a deposit by
 *     address of single contributions (Z < 64); if the grouping
 *     cannot be set up (no memory for its buffer), the forward runs without
 *     it.  Holds one buffer of 16 B per lookup per stream (see "Memory").
 * Shared array.  `shared` holds M elements of the storage type named by
 *   pss_hash_params.weight_dtype (float32, or bfloat16 bit patterns).
 *   Arithmetic is float32 throughout; bfloat16 values are widened exactly on
 *   load and rounded to nearest-even once per update.
 * Memory.  Every array argument is device memory owned by the caller; the
 *   library keeps no pointer after the call returns other than in the work it
 *   enqueued, and the indices and offsets pointers that identify a prepared
 *   grouping (compared by the next backward, never dereferenced by it).
 *   Scratch space of the backward and sparse-gradient calls is a
 *   library-owned device buffer kept per (device, stream) between calls and
 *   grown to the largest call made on that stream (taken from a
 *   library-owned memory pool), and so does a forward call with
 *   PSS_PREPARE_BACKWARD (with a library stream and two events when the
 *   grouping runs on the library's stream);
 *   pss_release_scratch returns all of these.
 *   While `stream` is being captured into a graph, scratch is allocated
 *   stream-ordered from the pool and freed on the same stream instead, so
 *   that the graph owns it.
 * Streams.  Work is enqueued on `stream` (0 = the legacy default stream) of
 *   the current device; calls return once the work is enqueued.
 * Errors.  Arguments are checked on the host before anything is enqueued; a
 *   violation returns PSS_ERR_INVALID_ARG (or PSS_ERR_UNSUPPORTED) and
 *   enqueues nothing.  A failed launch or runtime call returns PSS_ERR_HIP.
 *   Contents of device arrays (offsets monotone, indices in range) are
 *   preconditions that are not checked on the device; whatever they hold,
 *   every address the kernels touch stays inside the arrays described above
 *   (hash addresses are reduced mod M; item ranges are clamped to [0, N]).
 * Threads.  Concurrent calls on different streams are safe; calls made on one
 *   stream from several threads at once are enqueued one after the other.
 */
#ifndef PSS_H
#define PSS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PSS_PRIME 2147483647u /* p = 2^31 - 1 */
#define PSS_MAX_DIM 4096      /* largest embedding width d */

typedef enum { PSS_F32 = 0, PSS_BF16 = 1 } pss_dtype;

enum {
  PSS_OK = 0,
  PSS_ERR_INVALID_ARG = 1,
  PSS_ERR_UNSUPPORTED = 2,
  PSS_ERR_HIP = 3,
  PSS_ERR_NO_MEMORY = 4,
  PSS_ERR_SCRATCH_LIMIT = 5  /* pss_backward_update_noalloc: more scratch needed
                                than PSS_NOALLOC_SCRATCH_BYTES */
};

/* Bytes of the static device scratch of pss_backward_update_noalloc (each
 * GPU the library runs on holds one such array until the process ends). */
#define PSS_NOALLOC_SCRATCH_BYTES (64u << 20)

/* Backward variant, bits 0-1 of pss_hash_params.flags.
 *   AUTO    library's choice for the shape: SPARSE when the update is not
 *           fused (Adagrad, or bfloat16 storage) and M > 16 * N * d (low
 *           compression: a pass over all of M would dominate), else SORTED
 *           (by address for short chunks on an array held in HBM, see
 *           PSS_DEPOSIT_BY_ADDRESS).
 *   ATOMIC  every (lookup, dim) contribution added with a float atomic, into
 *           `shared` (SGD on float32 storage) or into a float32 gradient
 *           buffer followed by one streaming optimizer pass.
 *   SORTED  lookups are grouped by token (radix sort on the item hash), the
 *           output-gradient rows of each token are summed in registers, and
 *           each token's sum is added once at its hashed addresses (float
 *           atomics; a token whose lookups span several of the 256-pair
 *           pieces of the grouped order adds one partial sum per piece).
 *   SPARSE  Alg. 1 sparse branch: the unique locations and summed values of
 *           pss_gradient_sparse, then the optimizer applied at those
 *           locations only.  No float atomics: bit-identical run to run.
 *           Requires N * (d/Z) < 2^31.
 * ATOMIC and SORTED sum in no fixed order (SORTED with PSS_DEPOSIT_BY_ADDRESS
 * and Z >= 64 in a fixed one); all variants compute the same G up to float
 * rounding. */
enum { PSS_BWD_AUTO = 0, PSS_BWD_ATOMIC = 1, PSS_BWD_SORTED = 2, PSS_BWD_SPARSE = 3 };
#define PSS_BWD_MASK 3u

/* Options, bits 2-8 of pss_hash_params.flags (see "Options" above). */
#define PSS_SIGN_PM1 (1u << 2)
#define PSS_SIGN_SPARSE (2u << 2)
#define PSS_SIGN_MASK (3u << 2)
#define PSS_POOL_MEAN (1u << 4)
#define PSS_INDEX_I32 (1u << 5)
#define PSS_ROWS_BF16 (1u << 6)
#define PSS_PREPARE_BACKWARD (1u << 7)
/* Bit 8: the deposit of the SORTED variant (or of AUTO) is ordered by
 * address instead of grouped by token (see PSS_DEPOSIT_BY_ADDRESS above). */
#define PSS_DEPOSIT_BY_ADDRESS (1u << 8)
#define PSS_FLAGS_ALL 0x1ffu

typedef struct {
  uint32_t a;            /* hash multiplier, 1 <= a <= p - 1 */
  uint32_t b;            /* hash offset,     0 <= b <= p - 1 */
  uint32_t num_tables;   /* T >= 1 */
  uint32_t batch;        /* B >= 1 (bags = T*B, table-major) */
  int64_t num_indices;   /* N = number of entries of `indices` (= offsets[T*B]) */
  int32_t weight_dtype;  /* pss_dtype of `shared` */
  float eps;             /* Adagrad epsilon (ignored by SGD); >= 0 */
  uint32_t flags;        /* PSS_BWD_* in bits 0-1, options in bits 2-8; the
                            sign field value 3 << 2 and bits 9 and up are
                            invalid */
  uint32_t sign_a;       /* sign hash multiplier, 1 <= sign_a <= p - 1
                            (read only when a sign option is set) */
  uint32_t sign_b;       /* sign hash offset, 0 <= sign_b <= p - 1 */
} pss_hash_params;

/* Fills p->a, p->b, p->sign_a and p->sign_b from `seed` (other fields
 * untouched): with x1 .. x4 the first four outputs of SplitMix64 (Steele,
 * Lea & Flood 2014) started from state `seed`, a = 1 + (x1 mod (p - 1)),
 * b = x2 mod p, sign_a = 1 + (x3 mod (p - 1)), sign_b = x4 mod p.  Host
 * only.  Returns PSS_ERR_INVALID_ARG if p is NULL. */
int pss_hash_params_from_seed(uint64_t seed, pss_hash_params* p);

/* Forward: pooled embeddings (paper Sec. 2.4 forward, Sec. 2.5 mapping).
 *   out[b][t*d + j*Z + k] = sum over e in bag t*B+b of
 *                           s(e, j) * shared[(h(indices[e], t, j) + k) mod M]
 *   (s = 1 without a sign option; divided by |bag| with PSS_POOL_MEAN)
 * shared   device, M elements of hash_params->weight_dtype, read only
 * M        1 <= M <= p;  Z: 1 <= Z <= M;  d: 1 <= d <= 4096, Z divides d
 * indices  device int64[N];  offsets: device int64[T*B + 1] (int32 each with
 *          PSS_INDEX_I32)
 * out      device float32[B][T*d] (bfloat16 with PSS_ROWS_BF16), fully
 *          overwritten; must not alias inputs
 * T*(d/Z) must be below 2^32. */
int pss_forward(const void* shared, int64_t M, int32_t Z, int32_t d,
                const pss_hash_params* hash_params, const void* indices,
                const void* offsets, void* out, hipStream_t stream);

/* The grouping step of the backward's SORTED variant (paper Alg. 1: the
 * lookups of a batch gathered by token before their gradients are summed),
 * started ahead of the backward: what PSS_PREPARE_BACKWARD makes pss_forward
 * do, as a call of its own, so that a caller can start it as soon as a
 * batch's indices and offsets are ready (before the forward call, or
 * without one).  It records an event on `stream` (everything enqueued there
 * before this call completes before the grouping reads indices and
 * offsets) and runs the grouping on a library-owned stream; the next
 * pss_backward_update on `stream` uses it under the conditions given for
 * PSS_PREPARE_BACKWARD, and the caller must not change the contents of
 * indices or offsets until then.  Arguments as for pss_forward (the
 * PSS_PREPARE_BACKWARD bit of hash_params->flags is not needed).  Does
 * nothing and returns PSS_OK while `stream` is being captured into a graph,
 * for N = 0 and for an explicit ATOMIC or SPARSE variant.  Returns
 * PSS_ERR_NO_MEMORY or PSS_ERR_HIP if the grouping could not be set up (the
 * backward then groups the batch itself). */
int pss_prepare_backward(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                         const void* indices, const void* offsets, hipStream_t stream);

/* Backward + optimizer step, in place (paper Sec. 2.4 backward, Alg. 1).
 *   G[m] = sum of s(e, j) * grad_out[b][t*d + j*Z + k] (divided by |bag| with
 *          PSS_POOL_MEAN) over every (item e, j, k) whose address
 *          (h + k) mod M equals m and whose chunk is read (s != 0)
 *   state == NULL : SGD       shared[m] -= lr * G[m]
 *   state != NULL : Adagrad   state[m] += G[m]^2;
 *                             shared[m] -= lr * G[m] / (sqrt(state[m]) + eps)
 * Every element that no lookup reads keeps its exact bits.  shared: device, M elements, updated in place.
 * state: device float32[M] or NULL, updated in place.  grad_out: device
 * float32[B][T*d] (bfloat16 with PSS_ROWS_BF16), read only.  Other arguments
 * as for pss_forward.  The SPARSE variant requires N * (d/Z) < 2^31 (else
 * PSS_ERR_UNSUPPORTED). */
int pss_backward_update(void* shared, float* state, int64_t M, int32_t Z, int32_t d,
                        const pss_hash_params* hash_params, const void* indices,
                        const void* offsets, const void* grad_out, float lr,
                        hipStream_t stream);

/* pss_backward_update for callers that cannot allocate memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, checks, variants and results, but every scratch buffer
 * (the float32 gradient buffer of an unfused update, the SORTED grouping,
 * the SPARSE workspace) lives in one static device array of
 * PSS_NOALLOC_SCRATCH_BYTES per GPU, and the call makes no allocation of
 * any kind (no hipMalloc, hipFree, pool or library allocation).  A call whose
 * scratch would exceed that size returns PSS_ERR_SCRATCH_LIMIT before
 * anything is enqueued: the SORTED grouping takes 16 B per lookup plus
 * about 0.5 B per lookup of digit counts (the headline one-hot batch of 1.7M
 * lookups needs 28 MB), an unfused update adds 4 B per weight of M.  A call
 * neither uses nor drops a grouping prepared by pss_prepare_backward or
 * PSS_PREPARE_BACKWARD.  Every call on one GPU shares that GPU's array and
 * leaves its contents behind (each call clears what it reads before
 * writing): calls that overlap in time on one GPU (different streams, or
 * host threads without ordering) race on it and must be ordered by the
 * caller.  The device address of the array is looked up on the first call
 * on each device (with that device current). */
int pss_backward_update_noalloc(void* shared, float* state, int64_t M, int32_t Z, int32_t d,
                                const pss_hash_params* hash_params, const void* indices,
                                const void* offsets, const void* grad_out, float lr,
                                hipStream_t stream);

/* Sparse gradient of the shared array (paper Alg. 1, sparse branch:
 * findUnique over the read locations, scatter_add of the output gradient):
 *   locations[0 .. U)  the distinct elements m of `shared` that at least one
 *                      (lookup, dim) reads, ascending (uint32, m < M)
 *   values[k]          sum of grad_out over every (lookup, dim) reading
 *                      locations[k], float32, summed in a fixed order
 *   *num_unique        U (int64, device memory)
 * The same G as the dense gradient at those locations.  capacity: length of
 * the caller's locations/values arrays (device); must be at least
 * min(M, N*d), else PSS_ERR_INVALID_ARG.  Requires N * (d/Z) < 2^31 (else
 * PSS_ERR_UNSUPPORTED).  Other arguments and options as for
 * pss_backward_update (an element read only by chunks of factor 0 is not a
 * location); nothing is updated.  Bit-identical from run to run. */
int pss_gradient_sparse(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const void* indices, const void* offsets, const void* grad_out,
                        uint32_t* locations, float* values, int64_t capacity, int64_t* num_unique,
                        hipStream_t stream);

/* Writes h(indices[e], t(e), j) for every item e and chunk j:
 * base_out: device uint32[N][d/Z].  Same arguments and checks as pss_forward;
 * exists so that hashed addresses can be compared bit for bit. */
int pss_debug_addresses(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const void* indices, const void* offsets, uint32_t* base_out,
                        hipStream_t stream);

/* Writes the chunk factor s(e, j) (+1, -1 or 0; +1 for every chunk when no
 * sign option is set) for every item e and chunk j: sign_out: device
 * int8[N][d/Z].  Same arguments and checks as pss_debug_addresses; the
 * kernels evaluate the sign hash from the item hash, this export lets it be
 * compared bit for bit with the definition. */
int pss_debug_signs(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                    const void* indices, const void* offsets, int8_t* sign_out,
                    hipStream_t stream);

/* Timing hook for measurement tools (no part of the method).  With two
 * non-null events (hipEvent_t, created by the caller with timing enabled and
 * kept alive while the hook is set), every later backward call that runs
 * the sorted path's reduce-and-deposit kernel launches it so that its
 * dispatch records `before` when the kernel starts and `after` when it ends:
 * hipEventElapsedTime then gives the kernel's own duration, without the
 * wait for earlier work on the stream or the dispatch.  Two nulls switch it
 * off; one null and one event is PSS_ERR_INVALID_ARG.  One setting for the
 * whole process: meant for one caller timing its own calls outside graph
 * capture, not for concurrent callers. */
int pss_debug_reduce_events(void* before, void* after);

/* Host evaluation of the same hash code the kernels run (no GPU needed):
 * base_out[e*C + j] = h(indices[e], t(e), j) for host arrays indices[N],
 * offsets[T*B+1] (int64 whatever the flags say) and base_out[N*C].  Returns
 * PSS_ERR_INVALID_ARG on bad arguments or on offsets that are not a valid
 * partition of [0, N). */
int pss_hash_bases_host(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const int64_t* indices, const int64_t* offsets, uint32_t* base_out);

/* Host evaluation of the chunk factors, through the same route as the
 * kernels (second hash from the item hash): sign_out[e*C + j] = s(e, j) for
 * host arrays as in pss_hash_bases_host and sign_out[N*C] (int8). */
int pss_hash_signs_host(int64_t M, int32_t Z, int32_t d, const pss_hash_params* hash_params,
                        const int64_t* indices, const int64_t* offsets, int8_t* sign_out);

/* Host check of a host copy of offsets: offsets[0] == 0, non-decreasing,
 * offsets[T*B] == N.  Returns PSS_OK or PSS_ERR_INVALID_ARG. */
int pss_validate_offsets_host(const int64_t* offsets, int64_t num_bags, int64_t N);

/* Frees the scratch buffers kept between calls, the streams, events and
 * buffers of PSS_PREPARE_BACKWARD and the library's memory pools (see
 * "Memory" above), on every device that holds them, after waiting for that
 * device's work to finish.  Host only; no call of this library may be in
 * progress on another thread.  Later calls allocate afresh; a prepared
 * grouping not yet used is dropped.  A program should call it before the
 * HIP runtime shuts down (the Python binding does so at interpreter exit),
 * so that the runtime's own teardown finds no library-owned object left.
 * Returns PSS_ERR_HIP if a runtime call fails (everything is forgotten
 * either way). */
int pss_release_scratch(void);

/* Static, NUL-terminated description of a status code. */
const char* pss_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* PSS_H */

/*
 * netkv.h -- C ABI of libnetkv, NetKV decode-instance selection on MI355X.
 *
 * Method: "NetKV: Network-Aware Decode Instance Selection for Disaggregated
 * LLM Inference".  For a request that finished prefill on instance p, every
 * decode instance d is scored with Eq. (5):
 *     C(d) = s_eff(d) / B_eff(p,d) + L_tau          (Eqs. (3), (4))
 *          + alpha * (T_queue(d) + T_decode(d))      (Sec. IV-B, Eqs. (6)-(7))
 * with s_eff(d) = bpt * (l_r - B_tok * j) (Eq. (2), j = leading blocks of the
 * request's hash run resident on d, Sec. III-B) under the memory feasibility
 * mask m_d >= s_eff(d) + m_min (Eq. (5) feasible set), and the minimum-cost
 * feasible d is selected, ties to the lowest index (Algorithm 1).  A batch of
 * requests is scored against one telemetry snapshot; the in-flight counter
 * update of Algorithm 1 is applied between batches (netkv_commit_batch).
 *
 * Conventions for every call:
 *   - Returns NETKV_OK (0) or a negative status; netkv_last_error(h) gives
 *     the message of the last failing call on h.
 *   - Every argument is validated before anything is launched, so a call
 *     that returns an error has written no output.
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *   - Units: bytes, seconds, bytes per second.
 *   - A handle is used by one host thread at a time; handles are independent.
 *   - Output bytes are identical from run to run (no floating-point atomics;
 *     reductions are minima over packed (score, index) keys).
 */
#ifndef NETKV_H
#define NETKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct netkv_ctx *netkv_handle;
typedef int32_t netkv_status;

enum {
    NETKV_OK = 0,
    NETKV_EINVAL = -1,     /* bad argument or bad input values */
    NETKV_ENOTREADY = -2,  /* select/sweep/commit before both loads */
    NETKV_ENOMEM = -3,     /* device allocation failed */
    NETKV_EDEVICE = -4,    /* a HIP runtime error */
    NETKV_ECAPACITY = -5   /* a resident-set table cannot be built */
};

/* Create a handle bound to HIP device `device`.  *out receives the handle. */
netkv_status netkv_create(netkv_handle *out, int device);

/* Release the handle and every device buffer it owns (waits for its work). */
void netkv_destroy(netkv_handle h);

/* Message of the last failing call on h (empty string if none; never NULL).
 * The string stays valid until the next call on h. */
const char *netkv_last_error(netkv_handle h);

/*
 * One telemetry snapshot: the network cost oracle's maps (Sec. III-E:
 * tier map, tier bandwidth, tier latency, congestion) plus the scheduler's
 * view of decode state (Sec. III-C) and the cost-model parameters.
 * Array pointers may be host or device memory; they are copied.
 */
typedef struct {
    uint32_t n_prefill, n_decode;   /* P >= 1, D >= 1 */
    const uint8_t *tier_map;        /* [P*D], row-major by prefill: tau(p,d) in 0..3 */
    const float *util;              /* [P*D] congestion c(p,d) in [0,1) for the pair's tier
                                       (per-pair form of the per-tier c_tau) */
    double tier_bw[4];              /* B_k > 0, bytes/s (the oracle's Gbps / 8 * 1e9) */
    double tier_lat[4];             /* L_k >= 0, seconds (the oracle's microseconds * 1e-6) */
    const uint16_t *n_inflight;     /* [4*P], tier-major: n_inflight[tau*P + p] (Eq. (4)) */
    const uint64_t *free_mem;       /* [D] m_d, bytes */
    const uint32_t *queue_depth;    /* [D] q_d */
    const uint32_t *batch_size;     /* [D] beta_d <= beta_max */
    double t_iter_a, t_iter_b;      /* t_iter(beta) = a + b*beta, seconds (Sec. III-C), >= 0 */
    uint32_t beta_max;              /* maximum batch size (Sec. IV-B) */
    double alpha;                   /* weight of T_queue + T_decode; 1 is Eq. (5) exactly, >= 0 */
    uint64_t m_min;                 /* per-instance memory reserve, bytes (Eq. (5)) */
    uint64_t kv_bytes_per_token;    /* per prefill/decode GPU pair (Eq. (1) / TP), < 2^32 */
    uint32_t block_tokens;          /* B_tok >= 1, tokens per hashed block (Sec. III-B) */
} netkv_oracle_t;

/* Load a snapshot (synchronous: returns after the copy and validation are
 * complete on `stream`, so the caller may free its arrays on return).
 * Also resets the between-batch state (n_inflight, queue_depth, free_mem
 * from the snapshot; admitted bytes of the previous batch to 0).
 * EINVAL: NULL pointer, P or D zero, P * (D + 32) >= 2^29, tier > 3, util outside [0,1) or NaN,
 * beta_d > beta_max, non-positive or non-finite bandwidth, negative or
 * non-finite latency/a/b/alpha, block_tokens 0, kv_bytes_per_token >= 2^32,
 * or D different from a loaded cache. */
netkv_status netkv_oracle_load(netkv_handle h, const netkv_oracle_t *o, void *stream);

/* Replace only the congestion matrix util [P*D] of the loaded snapshot
 * (a refreshed or stale congestion map; Sec. V-D).  Synchronous; host or
 * device pointer.  EINVAL for values outside [0,1) or NaN; ENOTREADY with
 * no snapshot loaded. */
netkv_status netkv_oracle_set_util(netkv_handle h, const float *util, void *stream);

/* Predictive congestion (Sec. VIII, future work: a lightweight time-series
 * prediction over the telemetry history in place of the instantaneous
 * snapshot, relying on the staleness tolerance of Proposition 2).  Reading:
 * simple exponential smoothing.  Each call folds one observation into the
 * handle's congestion matrix, which later selections use as their
 * forecast:
 *     c(p,d) <- c(p,d) + beta * (obs(p,d) - c(p,d)),   0 < beta <= 1,
 * in fp32; the first forecast is the loaded snapshot's (or the last
 * netkv_oracle_set_util) matrix, and beta = 1 takes the observation as is.
 * obs: DEVICE f32[n_prefill * n_decode], row-major by prefill.
 * Asynchronous on `stream`; allocates nothing.  An observation outside
 * [0, 1) or NaN leaves its entry unchanged and is reported by
 * netkv_sync_errors.  EINVAL: NULL obs, beta outside (0, 1]; ENOTREADY: no
 * snapshot loaded. */
netkv_status netkv_congestion_smooth(netkv_handle h, const float *obs, float beta, void *stream);

/* Copy the congestion matrix the selections currently use (snapshot, set,
 * or smoothed) to out: DEVICE f32[n_prefill * n_decode].  Asynchronous. */
netkv_status netkv_congestion_get(netkv_handle h, float *out, void *stream);

/* Load the resident block-hash sets K_d (Sec. III-B, III-C) of n_decode
 * decode instances as CSR: the hashes of decode d are
 * hashes[hash_off[d] .. hash_off[d+1]), n_hashes = hash_off[n_decode].
 * Host or device pointers.  Value 0 is reserved (EINVAL); repeated hashes
 * of one decode are allowed and count once.  Builds the holder index: one
 * open-addressed set of every distinct resident hash, with at most
 * `max_load_factor` (0 < lf < 1) occupancy (capped at 0.85; a build that
 * cannot place every hash is retried with twice the buckets, twice), and
 * for each hash its holders -- one decode, or a bitmap over the decodes
 * (8 * ceil(ceil(n_decode / 64) / 12) * 12 bytes per hash held by two or more) -- so
 * that one lookup answers a membership test on every decode at once.
 * Synchronous; needs about 28 bytes of temporary device memory per
 * resident hash while building.  EINVAL: bad CSR, hash 0, lf out of range,
 * D different from a loaded snapshot; ECAPACITY: 2^31 or more resident
 * hashes, a set of more than 2^31 slots, or one that could not be built
 * even at four times the planned buckets; ENOMEM: out of device memory. */
netkv_status netkv_cache_load(netkv_handle h, uint32_t n_decode, const uint64_t *hash_off,
                              const uint64_t *hashes, uint64_t n_hashes, float max_load_factor,
                              void *stream);

/* A batch of requests (DEVICE pointers), Sec. III-B: request r finished
 * prefill on instance prefill[r] < P, has l_r = len_tokens[r] >= 1 input
 * tokens and the block-hash run hashes[hash_off[r] .. hash_off[r+1]) of
 * length n_r = floor(l_r / B_tok), block 0 first; n_hashes bounds the
 * hashes array.  A request violating this is answered with index -1 and
 * score NaN and is reported by netkv_sync_errors. */
typedef struct {
    uint32_t n_req;
    const uint32_t *prefill;        /* [n_req] */
    const uint32_t *len_tokens;     /* [n_req] */
    const uint64_t *hash_off;       /* [n_req + 1] */
    const uint64_t *hashes;         /* [n_hashes]; a block hash 0 is resident
                                       on no decode (resident sets cannot
                                       hold 0), so a run's match ends there */
    uint64_t n_hashes;
} netkv_requests_t;

/* Optional per-pair outputs, row-major [n_req][n_decode] DEVICE arrays;
 * any member may be NULL. */
typedef struct {
    uint16_t *prefix_blocks;        /* j: leading resident blocks (lambda = B_tok * j),
                                       written as min(j, 65535) */
    uint8_t *feasible;              /* 1 iff m_d >= s_eff + m_min */
    float *score;                   /* C(r,d), also for infeasible pairs */
} netkv_pairs_t;

/* Score every (request, decode) pair and select, per request, the k
 * (1 <= k <= 8) feasible decodes of lowest cost in ascending (score, index)
 * order (the argmin of Algorithm 1 generalised to top-k); fewer than k
 * feasible decodes are padded with index -1 and score +inf (Algorithm 1
 * rejects a request with no feasible decode).  out_idx, out_score:
 * [n_req * k] DEVICE arrays.  `pairs` may be NULL.  Asynchronous on
 * `stream`: inputs must stay valid and outputs are defined once the stream
 * completes.  A batch of 2^16 requests or more also runs work on a second
 * stream of the handle, forked from `stream` and joined back to it by
 * events within the call, so ordering on `stream` (and a graph capture of
 * it) covers all of it.  Allocates only when a batch is
 * larger than the handle's work buffers hold -- every earlier batch's, or
 * what netkv_reserve sized them for -- and then grows them (about
 * 100 + 8*K*ceil(D/(64*C)) bytes per request, K the next power of two >= k
 * and C the decodes per lane, plus 4 bytes per block hash and the leader
 * table).
 * EINVAL: NULL pointers, k out of range; ENOTREADY: snapshot or cache
 * missing; n_req = 0 is a no-op. */
netkv_status netkv_select_batch(netkv_handle h, const netkv_requests_t *req, uint32_t k,
                                int32_t *out_idx, float *out_score, netkv_pairs_t *pairs,
                                void *stream);

/* netkv_select_batch in throughput mode (no per-pair outputs) without any
 * device allocation, for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, results and errors as netkv_select_batch with
 * pairs = NULL; the selections and scores are bit-identical to it.  Its
 * work buffers come from one static array of 64 MiB per device, part of the
 * library's device code, held from the device's first netkv_create until
 * the process ends.  A batch larger than the array holds (more than 65,536
 * requests, or fewer when k * ceil(n_decode / 64) is large) is processed
 * in consecutive sub-batches on `stream`, which is exact: every request's
 * result depends only on that request.  Leaders beyond the table the
 * array leaves room for are matched on their own (slower, same results).
 * Every call on a device shares that device's array and leaves its last
 * contents there: calls that overlap on one device (different streams or
 * threads, with no ordering between them) race and give undefined
 * results.  ECAPACITY when not even a sub-batch of 256 requests fits (a
 * pool of several million decodes); otherwise as netkv_select_batch. */
netkv_status netkv_select_batch_noalloc(netkv_handle h, const netkv_requests_t *req, uint32_t k,
                                        int32_t *out_idx, float *out_score, void *stream);

/* Size the handle's selection work buffers ahead for batches of up to
 * max_req requests with up to max_hashes block hashes and 1 <= k <= max_k,
 * so that netkv_select_batch, netkv_rank_sweep and netkv_select_sequential
 * allocate no work buffers for such batches afterwards (they grow them
 * otherwise, when a batch exceeds every earlier one) -- except the ranking
 * sweep's per-scenario factors (4 * n_scen * P * D bytes), which depend on
 * the scenario count.  Needs a loaded
 * snapshot (ENOTREADY) and is redone after a snapshot with another decode
 * count; synchronous with respect to allocation.  ENOMEM when the device
 * cannot hold them. */
netkv_status netkv_reserve(netkv_handle h, uint32_t max_req, uint64_t max_hashes, uint32_t max_k,
                           void *stream);

/* Two-hop KV routing (Sec. VIII, future work: KV state staged through an
 * intermediate cache in CPU DRAM or SSD; the oracle exposes both hops'
 * tiers and the cost sums the two transfer times).  Reading: every pair
 * (p, d) has, besides its direct route, a staged route p -> staging store
 * -> d whose hops have tiers tier1 / tier2 and congestion util1 / util2
 * (row-major [n_prefill * n_decode], like the snapshot's maps).  Its
 * transfer time is
 *     s_eff / B_eff(tier1, util1, n_inflight[tier1][p]) + L(tier1)
 *   + s_eff / B_eff(tier2, util2, 0) + L(tier2)
 * (the staging store's own transfers are not the prefill's in-flight ones;
 * Eqs. (3)-(4) per hop), and each pair's cost takes the faster of its two
 * routes (ties: direct).  Feasibility and the load term are unchanged, and
 * the policy rungs apply to both hops.  Only netkv_select_batch uses the
 * staged routes; the ranking sweep and the sequential form keep the direct
 * ones.  Synchronous; host or device pointers; the handle keeps copies
 * while the snapshot keeps its shape (a snapshot of another shape drops
 * them).  EINVAL: NULL map, tier > 3, util outside [0,1) or NaN (nothing is
 * changed); ENOTREADY: no snapshot loaded. */
netkv_status netkv_route2_load(netkv_handle h, const uint8_t *tier1, const float *util1,
                               const uint8_t *tier2, const float *util2, void *stream);

/* Drop the staged routes: selections score direct routes only again. */
netkv_status netkv_route2_clear(netkv_handle h);

/* The route of each selection under the current snapshot and route maps:
 * for idx[r*k + q] (DEVICE, as written by netkv_select_batch), out_route
 * (DEVICE int8[n_req * k]) = 1 when the staged route is strictly faster,
 * 0 when the direct one is (the scoring kernel's arithmetic), -1 for no
 * selection or an invalid request.  Asynchronous.  ENOTREADY: no route
 * maps, snapshot or cache loaded; EINVAL: k outside [1, 8], NULL arrays. */
netkv_status netkv_route2_of(netkv_handle h, const netkv_requests_t *req, uint32_t k,
                             const int32_t *idx, int8_t *out_route, void *stream);

/* Stale-telemetry ranking sweep (Sec. V-D, Proposition 2): re-rank the
 * batch under n_scen congestion scenarios util_scen [n_scen][P*D] (DEVICE,
 * each value in [0,1)).  Prefix matches do not depend on telemetry and are
 * computed once (the batch selection under the loaded snapshot, whose
 * leader rows give every pair's non-cached tokens).  Writes the top-k
 * (1 <= k <= 8) of every scenario to out_idx / out_score
 * [n_scen][n_req][k]; a scenario equal to the loaded congestion reproduces
 * netkv_select_batch's results bit for bit.  If out_flips is not NULL,
 * out_flips[2*s] = number of requests whose selected decode lies on a
 * different tier than the one selected under the loaded snapshot's own
 * congestion, out_flips[2*s+1] = number whose selected decode differs (a
 * rejection counts as its own tier and index).  If out_inversions is not
 * NULL, Proposition 2's quantity: over pairs of decodes on different tiers
 * from one prefill instance, with X = B'(1 - c), B' = B_tau / (1 +
 * n_inflight[tau][p]), under the snapshot's congestion and the scenario's,
 *   out_inversions[3*s]   = pairs the proposition covers: the larger of the
 *                           two pairs' congestion errors is below
 *                           |X - X'| / (B'_tau + B'_tau');
 *   out_inversions[3*s+1] = covered pairs whose order is inverted (0 by the
 *                           proposition);
 *   out_inversions[3*s+2] = all pairs whose strict snapshot order the
 *                           scenario does not keep;
 * evaluated in fp64 (the policy option does not apply to them).  For a
 * batch below 2^16 requests they run on the handle's second stream, forked
 * from `stream` and joined back to it by events before the call returns,
 * so ordering on `stream` (and a graph capture of it) covers them.
 * Asynchronous; grows internal buffers on first use (n_scen * P * D * 4
 * bytes of per-scenario factors, 16 bytes per request of records, and the
 * selection's buffers, see netkv_reserve).  Invalid requests get index -1
 * and score NaN in every scenario.  Scenario values are not validated
 * (values >= 1 give non-positive bandwidth and meaningless costs). */
netkv_status netkv_rank_sweep(netkv_handle h, const netkv_requests_t *req, uint32_t n_scen,
                              const float *util_scen, uint32_t k, int32_t *out_idx,
                              float *out_score, uint64_t *out_flips, uint64_t *out_inversions,
                              void *stream);

/* Between-batch update after the selections sel[n_req] (DEVICE; -1 =
 * rejected) of a batch (the in-flight increment of Algorithm 1 and the counter cap of
 * Sec. V-C, with one batch as the unit of time):
 *   n_inflight[tau][p] = min(cap, selections of the batch from p on tau);
 *   q_d = max(0, q_d + admitted_d - mu);
 *   m_d = max(0, m_d - A_d) + A_prev_d;  A_prev_d = A_d,
 * A_d = sum of s_eff over the requests admitted to d.  Integer arithmetic;
 * asynchronous.  EINVAL: NULL pointers or an index >= D in sel is reported
 * by netkv_sync_errors; ENOTREADY as for select. */
netkv_status netkv_commit_batch(netkv_handle h, const netkv_requests_t *req, const int32_t *sel,
                                uint32_t cap, uint32_t mu, void *stream);

/* Selections per tier (Sec. VII, the tier-shift statistic): counts[t] for
 * t = 0..3 = requests whose selected decode sel[r] (DEVICE, -1 = rejected)
 * lies on tier t from the request's prefill instance, counts[4] = rejected
 * requests.  counts: DEVICE u64[5], overwritten.  Asynchronous.  An index
 * >= D is not counted and is reported by netkv_sync_errors. */
netkv_status netkv_tier_counts(netkv_handle h, const netkv_requests_t *req, const int32_t *sel,
                               uint64_t *counts, void *stream);

/* Algorithm 1 applied request after request in batch order (Sec. V-A,
 * V-C): each request is scored with the in-flight counters as left by the
 * earlier requests of the batch from the same prefill instance, and its
 * selection increments n_inflight[tau(p, d*)][p] unless the counter has
 * reached `cap` (Sec. V-C default 16).  Requests of different prefill
 * instances do not interact.  Writes the argmin (index, score) per request
 * to out_idx / out_score ([n_req] DEVICE); invalid requests get -1 / NaN.
 * The handle's between-batch state is not changed (netkv_commit_batch
 * applies the batch).  Asynchronous.  The prefix lengths come from the
 * batch selection's per-request records and leader rows (no per-pair
 * buffer): the work buffers are netkv_select_batch's at k = 1 plus
 * 16 bytes per request (records by batch index) and 16 bytes per request
 * for the per-prefill ordering, grown when a batch exceeds every earlier
 * one (netkv_reserve sizes them ahead).  Runs of any length are valid. */
netkv_status netkv_select_sequential(netkv_handle h, const netkv_requests_t *req, uint32_t cap,
                                     int32_t *out_idx, float *out_score, void *stream);

/* Copy the between-batch state into caller arrays (host or device; any may
 * be NULL): n_inflight [4*P], queue_depth [D], free_mem [D],
 * admitted_prev [D].  Synchronous. */
netkv_status netkv_state_get(netkv_handle h, uint16_t *n_inflight, uint32_t *queue_depth,
                             uint64_t *free_mem, uint64_t *admitted_prev, void *stream);

/* Wait for `stream`, then report (and clear) input errors the kernels found
 * in requests or selections since the last check: EINVAL with a message
 * naming the first kind of error, or NETKV_OK. */
netkv_status netkv_sync_errors(netkv_handle h, void *stream);

/* Kernel timing: when enabled, the library records HIP events on `stream`
 * around the one scoring kernel of each call -- the kernel of
 * netkv_select_batch that scores every pair and keeps each decode group's
 * top-k (not the ordering, prefix-length or merge kernels), the sweep
 * kernel of netkv_rank_sweep, the per-prefill kernel of
 * netkv_select_sequential, the smoothing kernel of netkv_congestion_smooth
 * -- without synchronising.  netkv_kernel_ms waits
 * for the last of them and returns the mean milliseconds over the launches
 * timed since timing was last enabled (the latest 256 when there were more);
 * ENOTREADY when there were none.  Enabling creates the events (EDEVICE if
 * that fails) and restarts the count. */
netkv_status netkv_set_timing(netkv_handle h, int enable);
netkv_status netkv_kernel_ms(netkv_handle h, float *ms);

/* Tuning options (results never depend on them):
 *   NETKV_OPT_RUN_LEN -- requests per wavefront run in the batch order
 *                        (0 = automatic, else 1..2^20);
 *   NETKV_OPT_REUSE   -- 1 (default): prefix lengths are shared along an
 *                        order of the batch that makes requests with equal
 *                        leading blocks neighbours.  Only a "leader" -- a
 *                        request whose first block past the run it shares
 *                        with its predecessor is resident on some decode --
 *                        is matched from block 0; any other request takes,
 *                        on every decode, the smaller of its last leader's
 *                        prefix length and the shortest common run since
 *                        that leader (an exact identity);
 *                        0: common runs are taken as empty, so every
 *                        request whose block 0 is resident somewhere is
 *                        matched from block 0;
 *   NETKV_OPT_COLS    -- decodes per lane of a scoring wavefront: 0 =
 *                        automatic (the widest of 6, 3, 2 whose groups of
 *                        64 per lane-column split evenly over the 8 XCDs,
 *                        else 2 on pools of 256+ decodes, else 1), 1, 2,
 *                        3, 4, 6;
 *   NETKV_OPT_LEAD_CAP -- 0 (default): the leader table is sized by memory
 *                        (prefix lengths of at most 256 MiB); else at most
 *                        `value` leaders, and holder values of at most
 *                        `value` of their blocks, are kept per call.  A
 *                        request whose leader is not kept is matched from
 *                        block 0 on its own, and a leader whose blocks'
 *                        holder values are not kept looks them up itself.
 * and one option that does change results, selecting the rung of the
 * method's ablation (Sec. VI, Experiment 6) the costs use:
 *   NETKV_OPT_POLICY  -- 0 (default): the full cost; 1: static tier map and
 *                        self-contention counter, live congestion taken as 0;
 *                        2: static tier map only (congestion and in-flight
 *                        counters taken as 0). */
enum { NETKV_OPT_RUN_LEN = 1, NETKV_OPT_REUSE = 2, NETKV_OPT_COLS = 3, NETKV_OPT_POLICY = 4,
       NETKV_OPT_LEAD_CAP = 5 };
netkv_status netkv_set_option(netkv_handle h, int option, uint32_t value);

/* Geometry of the loaded cache's holder index (any pointer may be NULL):
 * slots of the hash set (two per bucket, a power of two of buckets),
 * distinct resident hashes, hashes resident on two or more decodes (one
 * bitmap row each), and device bytes of the set and the bitmaps.
 * ENOTREADY with no cache loaded. */
netkv_status netkv_cache_info(netkv_handle h, uint64_t *index_slots, uint64_t *distinct_hashes,
                              uint64_t *shared_hashes, uint64_t *index_bytes);

/* Non-cached bytes of each selection (Eq. (2), s_eff = bpt * (l_r -
 * B_tok * j) with j the selected pair's block prefix length, Sec. III-B):
 * for idx[r*k + q] (DEVICE, as written by netkv_select_batch) out_bytes
 * (DEVICE u64[n_req * k]) gets the bytes the transfer moves, 0 for no
 * selection or an invalid request.  The sizes of the KV transfers that
 * netkv_flow_sim takes.  Asynchronous; an index >= D is reported by
 * netkv_sync_errors.  ENOTREADY: no snapshot or cache; EINVAL: k outside
 * [1, 8], NULL arrays. */
netkv_status netkv_selection_bytes(netkv_handle h, const netkv_requests_t *req, uint32_t k,
                                   const int32_t *idx, uint64_t *out_bytes, void *stream);

/* Flow-level transfer simulation (Sec. VI-B, the evaluation simulator's
 * network model): KV transfers are flows over the links of their paths;
 * each link is shared max-min fairly among the flows crossing it, and every
 * flow arrival or completion re-evaluates the allocation of all flows in
 * progress.  Background traffic is a steady utilisation the caller takes
 * out of each link's capacity (the section's mean-field model).  The
 * allocation is computed by progressive filling: all unfrozen flows' rates
 * rise together until a link is full, and the flows crossing it stop
 * there.  fp64 throughout; results are bit-identical to a sequential
 * implementation of the same operations.
 *
 * n_inst independent instances, one workgroup each: instance i holds flows
 * flow_off[i] .. flow_off[i+1]-1 (n_flows = flow_off[n_inst] in all) on
 * links 0 .. n_links-1 with capacities cap[i * n_links + l] (bytes/s,
 * finite and > 0).  Flow f crosses the links path[path_off[f] ..
 * path_off[f+1]) (at least one, each < n_links, distinct within the flow;
 * n_path = path_off[n_flows]), moves bytes[f] >= 0 bytes and arrives at
 * start[f] (s, finite).  Writes finish[f], its completion time (s), and,
 * if stats is not NULL, stats[3i .. 3i+2] = the instance's allocations
 * computed (one per event), filling rounds over all of them, and flows in
 * progress summed over all of them.  All arrays DEVICE.  Asynchronous.
 * An instance with an invalid flow or capacity gets finish = NaN for all
 * its flows and is reported by netkv_sync_errors (as is one that reached an
 * iteration bound, which valid input never does); offsets that are not
 * non-decreasing, or that end past n_flows, make every instance invalid.
 * Each instance's flows are first sorted by arrival time (rocPRIM's
 * segmented radix sort), and the instances are started heaviest first (by
 * the sum over their flows of bytes over the least capacity on the path;
 * rocPRIM's radix sort), which only changes where each one runs.  Grows a
 * work buffer of the handle to 38 B per flow, 24 B per instance and the
 * two sorts' temporary storage, plus, for more
 * than 2,048 links (whose state then lives in device memory instead of
 * LDS), 17 B per link and instance.  EINVAL: NULL arrays, n_links = 0,
 * n_inst >= 2^31, n_flows >= 2^32. */
netkv_status netkv_flow_sim(netkv_handle h, uint32_t n_inst, uint32_t n_links, const double *cap,
                            const uint64_t *flow_off, uint64_t n_flows, const uint64_t *path_off,
                            const uint32_t *path, uint64_t n_path, const double *bytes, const double *start,
                            double *finish, uint64_t *stats, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* NETKV_H */

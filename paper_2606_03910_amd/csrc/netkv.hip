// libnetkv -- NetKV decode-instance selection for MI355X (gfx950).
//
// Host runtime and HIP kernels behind the C ABI declared in include/netkv.h.
// Method: "NetKV: Network-Aware Decode Instance Selection for Disaggregated
// LLM Inference", Algorithm 1 with Eqs. (2)-(7), evaluated for a whole batch
// of requests against one telemetry snapshot.
//
// Data layout in device memory (all owned by the handle):
//   * holder index of the resident block hashes of all decodes: every
//     distinct resident hash once in a two-choice bucketized cuckoo set
//     (two 8-byte slots per bucket, 0 = empty; hash value 0 is reserved),
//     with a 32-bit holder value per slot -- one decode, or a row of a
//     holder bitmap pool (one bit per decode).  One lookup answers a
//     membership test for every decode at once.
//   * snapshot: tier_map u8[P*D], util f32[P*D] (row-major by prefill),
//     n_inflight u16[4*P] (tier-major), free_mem u64[D], queue u32[D],
//     batch u32[D], plus the admitted bytes of the previous batch u64[D];
//     derived per call: (seconds per token, constant part) float2 rows per
//     prefill, and per decode the load term and feasibility limit.
//
// Kernels of one selection (netkv_select_batch), in launch order (a batch
// of 2^16 requests or more runs derive_kernel, then lead_holder_kernel and
// lead_kernel, on a second stream beside the others):
//   derive_kernel      -- per-call cost factors (Eqs. (3)-(7) split by what
//                         they depend on).
//   prep_kernel        -- validate requests, build hash-order keys.
//   sort kernels       -- stable radix sort into hash order (rocPRIM's for
//                         small and very large batches).
//   order_kernel       -- common leading run with the previous position,
//                         leaders (positions whose next block some decode
//                         holds), segmented-scan elements within each tile
//                         of positions, records.
//   tile_prefix_kernel -- the tiles' exclusive prefixes (the scan's second
//                         level).
//   lead_holder_kernel -- holder values of every leader's blocks.
//   sort kernels       -- stable sort into prefill order, writing the
//                         scoring records (or rocPRIM's sort and
//                         assemble_kernel).
//   lead_kernel        -- prefix lengths of every leader on every decode.
//   score_kernel       -- per pair: prefix length min(leader's, L*),
//                         feasibility and cost (Eqs. (2)-(7)), then the
//                         group's top-k; one wavefront per (run of requests,
//                         group of 64*C decodes); optional per-pair outputs.
//   reduce_kernel      -- merges the groups' keys into each request's top-k
//                         (not launched when one group covers the pool).
// Other calls:
//   derive_scen_kernel, sweep_kernel -- re-scoring under congestion
//                         scenarios from the leader rows; lanes over requests.
//   tier_inv_kernel    -- Proposition 2's tier-ranking inversion counts.
//   sequential kernels -- Algorithm 1's per-request in-flight increments,
//                         one workgroup per prefill instance, from the
//                         leader rows.
//   selection_bytes_kernel -- the selections' transfer sizes (Eq. (2)).
//   owner / classify / index_insert / index_value -- build the holder index.
// The flow-level transfer simulation is in flowsim.hip.
//   commit kernels     -- between-batch counter / queue / memory update.
#include <hip/hip_runtime.h>
#include <rocprim/device/device_radix_sort.hpp>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "netkv.h"
#include "netkv_internal.h"

namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr uint32_t kXcds = 8;   // accelerator complex dies of an MI355X, each with its own L2
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kMix64 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kEmptyKey = ~0ull; // empty top-k entry (sorts last)
// bytes of the static scratch array of the no-allocation selection (per device)
constexpr uint64_t kScratchBytes = 64ull << 20;

enum : uint32_t {
    kErrRequest = 1u,    // request header inconsistent
    kErrObservation = 2u,   // congestion observation outside [0, 1) or NaN
    kErrSelection = 4u,  // selection index out of range
    kErrTableFull = 8u,  // insertion found no free slot
    kErrFlow = kErrFlowBit,           // flow simulation: invalid flow set
    kErrFlowStall = kErrFlowStallBit,   // flow simulation: an iteration bound was reached
};

// ------------------------------------------------------------------ device data

struct Snap {
    const uint8_t *tier_map;
    const float *util;
    const uint16_t *n_inflight;
    const uint64_t *free_mem;
    const uint32_t *queue;
    const uint32_t *batch;
    float bw[4];
    float lat[4];
    float t_a, t_b, alpha;
    uint32_t beta_max;
    uint64_t m_min;
    uint32_t bpt;
    uint32_t block_tokens;
    uint32_t P, D;
    uint32_t policy;         // 0: full NetKV, 1: no live congestion, 2: neither congestion nor in-flight
    // derived once per call by derive_kernel (Eqs. (3)-(7) factored by (p, d) and d)
    const float2 *sl;        // [P][slp] per (p, d): seconds per non-cached token, and the
                             // constant part L_tau + alpha (T_queue + T_decode)
    uint32_t slp;            // row pitch of sl in elements (an odd number of 128-byte lines)
    const float2 *sr;        // like sl, for the staged (two-hop) route; null without one
    const float *dbase;      // [D] alpha (T_queue + T_decode)
    const uint64_t *dxlim;   // [D] x = l - lambda is feasible iff x < dxlim
};

// The holder index of the resident block hashes K_d of all decodes: every
// distinct resident hash once, in a bucketized two-choice cuckoo set (two
// candidate buckets of two 8-byte slots; 0 = empty), and in a parallel array
// the 32-bit holder value of the key in the same slot:
//   kHeldOne | d -- the hash is resident on decode d alone;
//   row          -- it is resident on two or more decodes, the set bits of
//                   row `row` of the bitmap pool (bit d % 64 of word d / 64).
// A hash that is not in the set is resident nowhere (kNoHolder).  One lookup
// answers a membership test for every decode at once.
constexpr uint32_t kHeldOne = 0x80000000u;
constexpr uint32_t kNoHolder = 0xFFFFFFFFu;

struct Table {
    const uint64_t *keys;   // [buckets][2] distinct resident hashes
    const uint32_t *vals;   // [buckets][2] holder values
    const uint64_t *bits;   // [rows][bpitch] holder bitmaps (at least one row, row 0 of zeros if unused)
    uint32_t shift;         // 64 - log2(buckets)
    uint32_t bpitch;        // 64-bit words per bitmap row, a multiple of 12
};

struct Reqs {
    uint32_t n_req;
    const uint32_t *prefill;
    const uint32_t *len;
    const uint64_t *off;
    const uint64_t *hashes;
    uint64_t n_hashes;
};

struct PairOut {
    uint16_t *j;        // [R][D]
    uint8_t *feas;      // [R][D]
    float *score;       // [R][D]
};

// The two candidate buckets of hash h in a set of 2^b buckets (shift =
// 64 - b): the top b bits of two 64-bit multiplicative hashes of the whole
// key (Fibonacci hashing, and the multiplier of splitmix64 after an
// xor-shift), the second xored onto the first with its low bit set, so the
// two buckets always differ.  Both use all 64 bits, so keys that agree in
// part of their bits still get independent bucket pairs.
__host__ __device__ inline void buckets_of(uint64_t h, uint32_t shift, uint32_t &b1, uint32_t &b2) {
    b1 = (uint32_t)((h * kGolden) >> shift);
    b2 = b1 ^ ((uint32_t)(((h ^ (h >> 31)) * kMix64) >> shift) | 1u);
}

// Row pitch (elements) of the per-(p, d) float2 rows: D rounded up to whole
// 128-byte lines, then to an odd number of lines, so that rows spread over
// all L2 sets instead of aliasing on the sets of a power-of-two stride.
__host__ __device__ inline uint32_t sl_pitch(uint32_t D) {
    uint32_t lines = (D + 15u) / 16u;
    if ((lines & 1u) == 0) ++lines;
    return lines * 16u;
}

// Elements allocated after the last row of the per-(p, d) rows and of the
// leaders' prefix-length table: one group of the widest scoring geometry
// (64 lanes x 6 decodes), so that the scoring kernel's loads for columns
// past the pool stay inside the allocation.
constexpr uint32_t kRowPad = 64u * 6u;

// Holder value of h, by one thread: both candidate buckets' keys, then the
// value of the slot that holds h (most looked-up hashes are held by no
// decode and need no value).
__device__ inline uint32_t holder_lane(const Table &t, uint64_t h) {
    if (h == 0) return kNoHolder;
    uint32_t b1, b2;
    buckets_of(h, t.shift, b1, b2);
    const ulonglong2 k1 = *(const ulonglong2 *)(t.keys + 2 * (uint64_t)b1);
    const ulonglong2 k2 = *(const ulonglong2 *)(t.keys + 2 * (uint64_t)b2);
    const uint64_t slot = k1.x == h ? 2 * (uint64_t)b1 : k1.y == h ? 2 * (uint64_t)b1 + 1
                        : k2.x == h ? 2 * (uint64_t)b2 : k2.y == h ? 2 * (uint64_t)b2 + 1 : ~0ull;
    return slot == ~0ull ? kNoHolder : t.vals[slot];
}

// Is h resident on decode d?
__device__ inline bool holds(const Table &t, uint64_t h, uint32_t d) {
    const uint32_t v = holder_lane(t, h);
    if (v == kNoHolder) return false;
    if (v & kHeldOne) return (v & ~kHeldOne) == d;
    return (t.bits[(uint64_t)v * t.bpitch + d / 64u] >> (d % 64u)) & 1ull;
}

// T_queue + T_decode of decode d, scaled by alpha (Sec. IV-B, Eqs. (6)-(7)).
__device__ inline float load_term(const Snap &s, uint32_t d) {
    int64_t q = (int64_t)s.queue[d];
    int64_t beta = (int64_t)s.batch[d];
    int64_t blocked = q - ((int64_t)s.beta_max - beta);
    blocked = blocked < 0 ? 0 : blocked;
    float t_cur = s.t_a + s.t_b * (float)beta;
    float t_next = s.t_a + s.t_b * (float)(beta + 1);
    return s.alpha * ((float)blocked * t_cur + t_next);
}

// The cost of Eq. (5) factored by what each factor depends on.  With
// x = l_r - lambda non-cached tokens (Eq. (2) divided by the bytes per token):
//   s_eff / B_eff(p,d) = x * bpt (1 + n_inflight[tau][p]) / (B_tau (1 - c(p,d)))
// (Eqs. (3)-(4)), so the pair contributes x * spt(p,d) + L_tau, and the decode
// alpha (T_queue + T_decode); feasibility m_d >= bpt x + m_min holds iff
// x < xlim_d = floor((m_d - m_min) / bpt) + 1 (integer, exact).
// Seconds per non-cached token with an explicit in-flight count n.  The
// ablation rungs of the method drop the live congestion (policy 1) or both
// the congestion and the in-flight term (policy 2).
__device__ inline float sec_per_token_n(const Snap &s, uint32_t tau, float n, float c) {
    const float ce = s.policy >= 1 ? 0.0f : c;
    const float ne = s.policy >= 2 ? 0.0f : n;
    return ((float)s.bpt * (1.0f + ne)) / (s.bw[tau] * (1.0f - ce));
}

__device__ inline float sec_per_token(const Snap &s, uint32_t tau, uint32_t p, float c) {
    return sec_per_token_n(s, tau, (float)s.n_inflight[tau * s.P + p], c);
}

// Tier latency by a per-lane tier index, without indexing an array.
__device__ inline float tier_latency(const Snap &s, uint32_t tau) {
    const float lo = (tau & 1u) ? s.lat[1] : s.lat[0];
    const float hi = (tau & 1u) ? s.lat[3] : s.lat[2];
    return (tau & 2u) ? hi : lo;
}

__device__ inline uint64_t feasible_limit(const Snap &s, uint64_t m) {
    if (m < s.m_min) return 0;
    if (s.bpt == 0) return ~0ull;
    return (m - s.m_min) / s.bpt + 1;
}

__device__ inline float pair_score(uint32_t x, float spt, float lat, float base) {
    return fmaf((float)x, spt, lat + base);
}

template <int K>
__device__ inline void topk_insert(uint64_t (&lst)[K], uint64_t x) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
        uint64_t lo = lst[i] < x ? lst[i] : x;
        x = lst[i] < x ? x : lst[i];
        lst[i] = lo;
    }
}

__device__ inline uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

// Index of the calling wavefront in its workgroup, as a wave-uniform value
// (so everything derived from it stays in scalar registers).
__device__ inline uint32_t wave_index() {
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

// Minimum of a 32-bit value over the 64 lanes with DPP row operations
// (quad permutes, row rotates, then the row broadcasts of wave64); every lane
// must be active.  The result is read from lane 63.
__device__ inline uint32_t wave_min_u32_dpp(uint32_t v) {
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x124, 0xF, 0xF, false));  // row_ror 4
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x128, 0xF, 0xF, false));  // row_ror 8
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x142, 0xA, 0xF, false));  // row_bcast 15
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x143, 0xC, 0xF, false));  // row_bcast 31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Minima over the 64 lanes of three values at once (12 VALU instructions
// where three wave_min_u32_dpp take 21).  permlane32_swap exchanges the
// upper half of a with the lower half of b, so one min leaves, in lanes
// 0-31, a's minimum over lanes l and l + 32 and, in lanes 32-63, b's.
// permlane16_swap then exchanges that register's odd rows of 16 lanes with
// c's even rows, and one min gives row 0 a's minimum over lanes i, i + 16,
// i + 32, i + 48, row 2 b's, and rows 1 and 3 c's over the lower and upper
// half.  A DPP minimum within each row finishes all of them: a in lane 0,
// b in lane 32, c the lesser of lanes 16 and 48.  Every lane must be
// active.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, CTRL, 0xF, 0xF, false);
}

__device__ inline void wave_min3_u32(uint32_t a, uint32_t b, uint32_t c, uint32_t &ma, uint32_t &mb,
                                     uint32_t &mc) {
    const auto s32 = __builtin_amdgcn_permlane32_swap(a, b, false, false);
    const uint32_t x = min((uint32_t)s32[0], (uint32_t)s32[1]);
    const auto s16 = __builtin_amdgcn_permlane16_swap(x, c, false, false);
    uint32_t z = min((uint32_t)s16[0], (uint32_t)s16[1]);
    z = min(z, dpp_u32<0xB1>(z));    // quad_perm 1,0,3,2
    z = min(z, dpp_u32<0x4E>(z));    // quad_perm 2,3,0,1
    z = min(z, dpp_u32<0x124>(z));   // row_ror 4
    z = min(z, dpp_u32<0x128>(z));   // row_ror 8
    ma = (uint32_t)__builtin_amdgcn_readlane((int)z, 0);
    mb = (uint32_t)__builtin_amdgcn_readlane((int)z, 32);
    mc = min((uint32_t)__builtin_amdgcn_readlane((int)z, 16), (uint32_t)__builtin_amdgcn_readlane((int)z, 48));
}

// Validate request r's header; returns false (and flags) if inconsistent.
__device__ inline bool request_ok(const Reqs &rq, const Snap &s, uint32_t r, uint32_t &p,
                                  uint32_t &len, uint64_t &a, uint32_t &n) {
    p = rq.prefill[r];
    len = rq.len[r];
    a = rq.off[r];
    uint64_t b = rq.off[r + 1];
    if (!(p < s.P && len >= 1 && b >= a && b <= rq.n_hashes)) return false;
    if (b - a != (uint64_t)(len / s.block_tokens)) return false;
    n = (uint32_t)(b - a);
    return true;
}

// Per-call factors of the cost: seconds per token and the constant part
// (tier latency plus load term) for every (p, d), the load term and the
// feasibility limit for every d.  Reads the current snapshot
// (congestion, in-flight counters, queue, batch, free memory).
__global__ __launch_bounds__(256) void derive_kernel(Snap s, float2 *__restrict__ sl, float *__restrict__ dbase,
                                                     uint64_t *__restrict__ dxlim) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t npd = (uint64_t)s.P * s.D;
    if (i < npd) {
        const uint32_t p = (uint32_t)(i / s.D);
        const uint32_t d = (uint32_t)(i - (uint64_t)p * s.D);
        const uint32_t tau = s.tier_map[i] & 3u;
        // the constant part is rounded exactly as latency + load term would
        // be when added after loading both (no contraction into an FMA)
        sl[(uint64_t)p * s.slp + d] =
            make_float2(sec_per_token(s, tau, p, s.util[i]), __fadd_rn(tier_latency(s, tau), load_term(s, d)));
    }
    if (i < s.D) {
        dbase[i] = load_term(s, (uint32_t)i);
        dxlim[i] = feasible_limit(s, s.free_mem[i]);
    }
}

// Two-hop routing (Sec. VIII): the staged route p -> staging store -> d of
// every pair, with hop tiers t1, t2 and congestion u1, u2.  Its transfer
// time is the sum of the hops' (Eqs. (3)-(4) each): seconds per token
// bpt (1 + n_inflight[t1][p]) / (B_t1 (1 - u1)) + bpt / (B_t2 (1 - u2)) (the
// staging store's transfers are not the prefill's in-flight ones) and the
// constant part L_t1 + L_t2 plus the decode's load term.
__global__ __launch_bounds__(256) void derive_route_kernel(Snap s, const uint8_t *__restrict__ t1,
                                                           const float *__restrict__ u1,
                                                           const uint8_t *__restrict__ t2,
                                                           const float *__restrict__ u2, float2 *__restrict__ sr) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t npd = (uint64_t)s.P * s.D;
    if (i >= npd) return;
    const uint32_t p = (uint32_t)(i / s.D);
    const uint32_t d = (uint32_t)(i - (uint64_t)p * s.D);
    const uint32_t a = t1[i] & 3u, b = t2[i] & 3u;
    const float spt = sec_per_token(s, a, p, u1[i]) + sec_per_token_n(s, b, 0.0f, u2[i]);
    sr[(uint64_t)p * s.slp + d] =
        make_float2(spt, __fadd_rn(__fadd_rn(tier_latency(s, a), tier_latency(s, b)), load_term(s, d)));
}

// ---------------------------------------------------------------- batch order
//
// Prefix lengths follow from a batch order that groups equal leading blocks.
// The sort key is 19 bits of the first block hash above 12 bits of the
// complemented run length, so requests that start with the same prefix are
// neighbours in descending length ("hash order").  For neighbours r' -> r
// with a common leading run of L blocks, the first-miss index of r on any
// decode d is j(r', d) whenever that lies inside the common run (blocks
// 0..j(r',d) of r are those of r'), and otherwise it is at least L.  So if
// block L of r is held by no decode (or r has no block L), j(r, d) =
// min(j(r', d), L) exactly, on every decode.
//
// A position whose block L some decode holds is a "leader": its prefix
// lengths are computed from block 0 on every decode (leader kernel).  Every
// other position m then has j(m, d) = min(j(ell, d), L*) with ell the last
// leader before it in hash order and L* the least common run L over the
// positions after ell up to m; with no leader before it, j = 0.  A
// segmented scan over the hash order gives each position its (ell, L*).
// Longest first, a request that is a prefix of its predecessor has L = n_r
// and one that leaves the shared chain first resumes at a block of its own,
// which usually no decode holds, so leaders are about one per shared chain.
//
// Scoring then runs in prefill order (the hash order kept within each
// prefill, a stable radix sort): consecutive requests share their row of
// the snapshot and often their leader, so both are re-read from L1.

constexpr uint32_t kKeyLenBits = 12;             // low key bits: 4095 - min(blocks, 4095)
constexpr uint32_t kKeyEmptyRun = 0x80000000u;   // valid request without blocks
constexpr uint32_t kKeyInvalid = 0xFFFFFFFFu;
constexpr uint32_t kNoLead = 0xFFFFFFFFu;        // no leader before the position
constexpr uint32_t kLeadOver = 0xFFFFFFFEu;      // a leader beyond the leader table's capacity
constexpr uint32_t kNoCap = 0xFFFFFFFFu;         // L* of a leader itself (no cap)

// Segmented-scan element of a hash-order position: leader slot (or kNoLead
// for a non-leader) in the high word, common run L (kNoCap for a leader) in
// the low word.  Combining keeps the later leader, else the earlier leader
// with the smaller L; the combination is associative.
__host__ __device__ inline uint64_t seg_elem(uint32_t slot, uint32_t l) { return ((uint64_t)slot << 32) | l; }
struct SegOp {
    __host__ __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
        if ((uint32_t)(b >> 32) != kNoLead) return b;
        const uint32_t la = (uint32_t)a, lb = (uint32_t)b;
        return (a & 0xFFFFFFFF00000000ull) | (la < lb ? la : lb);
    }
};

// The identity of SegOp: no leader, no cap.
constexpr uint64_t kSegIdentity = ((uint64_t)kNoLead << 32) | kNoCap;
__device__ inline uint64_t seg_op(uint64_t a, uint64_t b) { return SegOp()(a, b); }

// A leader: where its blocks' holder values start in hv (from block 0, up
// to the first block no decode holds; m = kNoPre if they did not fit), and
// its hash run for lookups otherwise.
struct alignas(16) Lead {
    uint64_t a;      // offset of the hash run
    uint64_t hoff;   // offset of the holder values
    uint32_t n;      // hashed blocks
    uint32_t m;      // stored holder values, or kNoPre
    uint32_t pad[2];
};
constexpr uint32_t kNoPre = 0xFFFFFFFFu;

// Token counts below 2^24 are integers that fp32 holds exactly: requests
// shorter than that are scored in fp32 with results identical to integer
// arithmetic, longer ones in integers.
constexpr uint32_t kExactTok = 1u << 24;

// A request by hash-order position: its prefill row and length.
struct Pre {
    uint32_t row;    // byte offset of the request's row of derived (p, d) values, p * slp * 8
    uint32_t len;    // input tokens
};

// One request in scoring order: the part every scoring step reads (one
// 16-byte scalar load) ...
struct alignas(16) Hot {
    uint32_t row;    // byte offset of the prefill row, as in Pre
    uint32_t lrow;   // byte offset of the leader's row of B_tok * j in the leader
                     // table; the all-zero row when there is no leader
    uint32_t len;    // input tokens, fp32 bits
    uint32_t lams;   // B_tok * L* (+inf for a leader itself), fp32 bits; negative:
                     // match this request on its own, in integers
};
constexpr uint32_t kHotPad = 2;   // records past the last position, read ahead by the scan

// ... and its index in the caller's batch (where its result goes, and its
// hash run and length when it is matched on its own).
struct Cold {
    uint32_t r;
};

struct Order {
    const Hot *hot;           // [n_valid + kHotPad] scoring-order request records
    const Cold *cold;         // [n_req]
    const float *lam;         // [leader rows][D] B_tok * prefix length of each leader on each decode
    const uint32_t *hv;       // holder values of the leaders' blocks
    const uint32_t *n_valid;  // valid requests (they sort first)
    uint32_t lead_cap;        // leaders the table takes in this call
};

// Validate each request and build its sort key, one thread per request.
// A request of more than max_blocks blocks is invalid (every call passes
// 2^32 - 1: runs of any length are scored).  A block hash 0 needs no
// check: no resident set holds it (cache loads reject it), so it is a miss
// on every decode, as the prefix definition gives.  vals (the input
// positions, for rocPRIM's sort) may be null.  Thread 0 clears the
// holder-value and leader counters of the order kernel.  An invalid
// request's outputs (index -1, score NaN) are written here when out_idx is
// given.
__global__ __launch_bounds__(256) void prep_kernel(Snap s, Reqs rq, uint32_t max_blocks, uint32_t *__restrict__ keys,
                                                   uint32_t *__restrict__ vals, uint32_t *__restrict__ err,
                                                   unsigned long long *__restrict__ hv_used,
                                                   unsigned int *__restrict__ n_lead, uint32_t k_out,
                                                   int32_t *__restrict__ out_idx, float *__restrict__ out_score) {
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r == 0) {
        *hv_used = 0;
        *n_lead = 0;
    }
    bool bad = false;
    if (r < rq.n_req) {
        uint32_t p, len, n;
        uint64_t a;
        const bool ok = request_ok(rq, s, r, p, len, a, n) && n <= max_blocks;
        uint32_t key = kKeyInvalid;
        if (ok) {
            if (n == 0) {
                key = kKeyEmptyRun;
            } else {
                const uint32_t top = (uint32_t)((rq.hashes[a] * kGolden) >> 32);
                key = ((top >> 13) << kKeyLenBits) | (4095u - (n < 4095u ? n : 4095u));
            }
        }
        keys[r] = key;
        if (vals) vals[r] = r;
        bad = !ok;
        if (bad && out_idx) {
            // an invalid request is answered here (the scoring kernel skips it)
            for (uint32_t q = 0; q < k_out; ++q) {
                out_idx[(uint64_t)r * k_out + q] = -1;
                out_score[(uint64_t)r * k_out + q] = __builtin_nanf("");
            }
        }
    }
    if (__ballot(bad) && (threadIdx.x % kWave) == 0) atomicOr(err, kErrRequest);
}

// Per hash-order position i (G lanes, G divides 64): the common leading run
// L with the previous position (G blocks compared per step, their loads
// issued together), whether the position is a leader (some decode holds its
// block L), and for a leader a slot of the leader table and room for the
// holder values of its blocks (in hv, from a shared counter; filled by
// lead_holder_kernel).  Writes the prefill sort key and the scoring record
// of i, and the number of valid requests (valid keys sort first): the last
// valid position writes it, or position 0 writes 0.  Invalid positions sort
// after every prefill (key P).
//
// The segmented scan of the positions' elements (leader slot, L) is fused
// here, in two levels: each workgroup (kOrderPos positions, one tile) scans
// its own elements and writes, for each position, the inclusive combination
// within the tile (seg) and the tile's total (agg[tile]).
// tile_prefix_kernel turns the totals into exclusive tile prefixes, and the
// record writers combine a position's tile prefix with its in-tile value.
// (A single-pass look-back over tiles was slower here: a tile's prefix can
// be published only a device-scope load round-trip after its predecessor's,
// far slower than tiles complete.)
constexpr uint32_t kLcpLanes = 4;                  // lanes per hash-order position
constexpr uint32_t kOrderPos = 256 / kLcpLanes;    // hash-order positions per order workgroup

// 64-bit lane shuffle up by `off` lanes (within the wavefront).
__device__ inline uint64_t shfl_up_u64(uint64_t v, uint32_t off) {
    const uint32_t lo = (uint32_t)__shfl_up((int)(uint32_t)v, off, kWave);
    const uint32_t hi = (uint32_t)__shfl_up((int)(uint32_t)(v >> 32), off, kWave);
    return ((uint64_t)hi << 32) | lo;
}

template <uint32_t G>
__global__ __launch_bounds__(256) void order_kernel(Reqs rq, uint32_t P, uint32_t slp, uint32_t bt,
                                                    const uint32_t *__restrict__ perm,
                                                    const uint32_t *__restrict__ sorted_keys, Table t,
                                                    uint32_t reuse, uint64_t *__restrict__ seg,
                                                    uint64_t *__restrict__ agg,
                                                    uint32_t *__restrict__ pkey, uint32_t *__restrict__ pval,
                                                    Pre *__restrict__ hrec, Cold *__restrict__ crec,
                                                    Lead *__restrict__ lead, uint32_t lead_cap,
                                                    unsigned int *__restrict__ n_lead, uint64_t hv_cap,
                                                    unsigned long long *__restrict__ hv_used,
                                                    uint32_t *__restrict__ n_valid) {
    static_assert(G * kOrderPos == 256, "positions per workgroup");
    __shared__ uint64_t wtot[kWavesPerBlock];
    const uint32_t sub = threadIdx.x % G;
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t seg0 = lane - sub;   // first lane of this position's lanes
    const uint64_t i = (uint64_t)blockIdx.x * kOrderPos + threadIdx.x / G;
    const bool inb = i < (uint64_t)rq.n_req;
    const bool valid = inb && sorted_keys[i] < kKeyInvalid;
    const uint32_t r = inb ? perm[i] : 0u;
    uint64_t e = kSegIdentity;   // this position's scan element (lane sub == 0)
    if (inb && sub == 0) {
        if (valid && (i + 1 == rq.n_req || sorted_keys[i + 1] >= kKeyInvalid)) *n_valid = (uint32_t)(i + 1);
        if (i == 0 && !valid) *n_valid = 0;
        if (pval) pval[i] = (uint32_t)i;
        if (!valid) {
            e = seg_elem(kNoLead, 0);
            pkey[i] = P;
            hrec[i] = Pre{0, 0};
            crec[i] = Cold{r};
        }
    }
    // this position's run, and the previous position's: from the lanes G
    // below (one wavefront holds kWave / G consecutive positions), or, for
    // the wavefront's first position, loaded
    uint64_t a = 0, nr = 0;
    if (valid) {
        a = rq.off[r];
        nr = rq.off[r + 1] - a;
    }
    const uint32_t pg = lane / G;
    const uint32_t key = valid ? sorted_keys[i] : kKeyInvalid;
    uint32_t kq = (uint32_t)__shfl_up((int)key, G, kWave);
    uint64_t b = shfl_up_u64(a, G), nq = shfl_up_u64(nr, G);
    if (pg == 0 && valid && i > 0) {
        kq = sorted_keys[i - 1];
        const uint32_t q = perm[i - 1];
        b = rq.off[q];
        nq = rq.off[q + 1] - b;
    }
    // keys that differ in their first-block hash bits have different first
    // blocks: nothing in common
    const bool cmp = valid && i > 0 && reuse && (key >> kKeyLenBits) == (kq >> kKeyLenBits);
    const uint64_t m = cmp ? (nr < nq ? nr : nq) : 0;
    uint64_t l = m;
    {
        // Lock-step over the wavefront: each lane loads U consecutive blocks
        // of its own run per step (their loads issued together) while its
        // position or the next one is still comparing, and takes the
        // previous position's blocks from the lanes G below; the first
        // differing block is the lowest lane's first stop.
        constexpr uint32_t U = 2;
        bool act = m > 0;
        for (uint64_t base = 0;; base += (uint64_t)G * U) {
            if (!__any(act)) break;
            const bool act_next = (bool)__shfl_down((int)act, G, kWave) && pg + 1 < (uint32_t)kWave / G;
            const bool need = act || act_next;
            const uint64_t x0 = base + (uint64_t)sub * U;
            uint64_t hr[U], hq[U];
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) hr[u] = (need && x0 + u < nr) ? rq.hashes[a + x0 + u] : 0ull;
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) hq[u] = shfl_up_u64(hr[u], G);
            if (pg == 0) {
#pragma unroll
                for (uint32_t u = 0; u < U; ++u) hq[u] = (act && x0 + u < m) ? rq.hashes[b + x0 + u] : 1ull;
            }
            uint32_t ls = U;   // this lane's first stop (U: none); blocks at m and beyond stop
#pragma unroll
            for (int u = (int)U - 1; u >= 0; --u)
                if (x0 + u >= m || hr[u] != hq[u]) ls = (uint32_t)u;
            const uint32_t bits =
                (uint32_t)(__ballot(act && ls < U) >> seg0) & (uint32_t)((1ull << G) - 1);
            if (act && bits) {
                const uint32_t fl = (uint32_t)__builtin_ctz(bits);
                const uint32_t lsf = (uint32_t)__shfl((int)ls, (int)(seg0 + fl), kWave);
                const uint64_t first = base + (uint64_t)fl * U + lsf;
                l = first < m ? first : m;
                act = false;
            }
            if (base + (uint64_t)G * U >= m) act = false;
        }
    }
    if (valid) {
        if (sub == 0) {
            // a leader if some decode holds block L
            const uint32_t vl = l < nr ? holder_lane(t, rq.hashes[a + l]) : kNoHolder;
            e = seg_elem(kNoLead, (uint32_t)l);
            if (vl != kNoHolder) {
                const unsigned int slot = atomicAdd(n_lead, 1u);
                if (slot >= lead_cap) {
                    e = seg_elem(kLeadOver, kNoCap);
                } else {
                    e = seg_elem(slot, kNoCap);
                    const unsigned long long o = atomicAdd(hv_used, (unsigned long long)nr);
                    Lead ld;
                    ld.a = a;
                    ld.hoff = o;
                    ld.n = (uint32_t)nr;
                    ld.m = o + nr <= hv_cap ? 0u : kNoPre;   // filled by lead_holder_kernel
                    ld.pad[0] = ld.pad[1] = 0;
                    lead[slot] = ld;
                }
            }
            pkey[i] = rq.prefill[r];
            hrec[i] = Pre{rq.prefill[r] * slp * (uint32_t)sizeof(float2),   // < 2^32 (checked at load)
                          rq.len[r]};
            crec[i] = Cold{r};
        }
    }
    // the tile's scan: the wavefront's positions (lanes sub == 0, G apart)
    // by shuffles, then the wavefronts' totals in order
#pragma unroll
    for (uint32_t off = G; off < (uint32_t)kWave; off <<= 1) {
        const uint64_t prev = shfl_up_u64(e, off);
        if (lane >= off) e = seg_op(prev, e);
    }
    const uint32_t w = threadIdx.x / kWave;
    if (lane == kWave - G) wtot[w] = e;
    __syncthreads();
    uint64_t pre = kSegIdentity;
    for (uint32_t q = 0; q < w; ++q) pre = seg_op(pre, wtot[q]);
    e = seg_op(pre, e);
    if (inb && sub == 0) seg[i] = e;
    if (threadIdx.x == 0) {
        uint64_t tot = kSegIdentity;
#pragma unroll
        for (uint32_t q = 0; q < kWavesPerBlock; ++q) tot = seg_op(tot, wtot[q]);
        agg[blockIdx.x] = tot;
    }
}

// Exclusive prefixes of the order workgroups' tile totals, in place: one
// workgroup of kPrefixThreads, kPrefixThreads * kPrefixPer totals per round
// (one round up to 2^24 requests), each thread combining its consecutive
// totals, the threads' results scanned by shuffles and then across the
// wavefronts, with the running prefix of earlier rounds.
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
constexpr uint32_t kPrefixThreads = 1024;
constexpr uint32_t kPrefixWaves = kPrefixThreads / kWave;
constexpr uint32_t kPrefixPer = 16;
static_assert(kPrefixPer % 2 == 0, "totals move in pairs");
__global__ __launch_bounds__(kPrefixThreads) void tile_prefix_kernel(uint64_t *__restrict__ agg, uint32_t n) {
    __shared__ uint64_t wtot[kPrefixWaves];
    __shared__ uint64_t carry_s;
    const uint32_t tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
    uint64_t carry = kSegIdentity;
    for (uint64_t r0 = 0; r0 < n; r0 += (uint64_t)kPrefixThreads * kPrefixPer) {
        const uint64_t b0 = r0 + (uint64_t)tid * kPrefixPer;
        // a thread's totals are consecutive: whole runs move in 16-byte
        // pieces (half the requests of 8-byte ones), the tail one by one
        const bool whole = b0 + kPrefixPer <= n;
        uint64_t v[kPrefixPer];
        if (whole) {
            const u64x2 *src = (const u64x2 *)(agg + b0);   // 16-byte aligned: b0 is a multiple of 16
#pragma unroll
            for (uint32_t u = 0; u < kPrefixPer / 2; ++u) {
                const u64x2 x = src[u];
                v[2 * u] = x.x;
                v[2 * u + 1] = x.y;
            }
        } else {
#pragma unroll
            for (uint32_t u = 0; u < kPrefixPer; ++u) v[u] = b0 + u < n ? agg[b0 + u] : kSegIdentity;
        }
        uint64_t tot = kSegIdentity;
#pragma unroll
        for (uint32_t u = 0; u < kPrefixPer; ++u) tot = seg_op(tot, v[u]);
        // inclusive scan of the threads' totals within the wavefront
        uint64_t inc = tot;
#pragma unroll
        for (uint32_t off = 1; off < (uint32_t)kWave; off <<= 1) {
            const uint64_t prev = shfl_up_u64(inc, off);
            if (lane >= off) inc = seg_op(prev, inc);
        }
        const uint64_t prev1 = shfl_up_u64(inc, 1);
        if (lane == kWave - 1) wtot[w] = inc;
        __syncthreads();
        uint64_t pre = carry;
        for (uint32_t q = 0; q < w; ++q) pre = seg_op(pre, wtot[q]);
        // this thread's first total's exclusive prefix
        uint64_t run = lane > 0 ? seg_op(pre, prev1) : pre;
        uint64_t ex[kPrefixPer];   // the exclusive prefixes
#pragma unroll
        for (uint32_t u = 0; u < kPrefixPer; ++u) {
            ex[u] = run;
            run = seg_op(run, v[u]);
        }
        if (whole) {
            u64x2 *dst = (u64x2 *)(agg + b0);
#pragma unroll
            for (uint32_t u = 0; u < kPrefixPer / 2; ++u) {
                u64x2 x;
                x.x = ex[2 * u];
                x.y = ex[2 * u + 1];
                dst[u] = x;
            }
        } else {
#pragma unroll
            for (uint32_t u = 0; u < kPrefixPer; ++u)
                if (b0 + u < n) agg[b0 + u] = ex[u];
        }
        if (tid == kPrefixThreads - 1) carry_s = run;
        __syncthreads();
        carry = carry_s;
        __syncthreads();
    }
}

// The scanned element (last leader slot, L*) of hash-order position i: its
// tile's exclusive prefix combined with its inclusive value in the tile.
__device__ inline uint64_t scanned_at(const uint64_t *seg, const uint64_t *tpre, uint64_t i) {
    return seg_op(tpre[i / kOrderPos], seg[i]);
}

// Holder values of every leader's blocks from block 0 up to the first
// block no decode holds: one wavefront per leader (looping over leaders,
// whose count is read from device memory), lanes over blocks.
__global__ __launch_bounds__(kBlock) void lead_holder_kernel(Table t, const uint64_t *__restrict__ hashes,
                                                             Lead *__restrict__ lead,
                                                             const unsigned int *__restrict__ n_lead,
                                                             uint32_t lead_cap, uint32_t *__restrict__ hv) {
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t nl_all = *n_lead;
    const uint32_t nl = nl_all < lead_cap ? nl_all : lead_cap;
    const uint32_t nw = gridDim.x * kWavesPerBlock;
    for (uint32_t slot = blockIdx.x * kWavesPerBlock + wave_index(); slot < nl; slot += nw) {
        const Lead ld = lead[slot];
        if (ld.m == kNoPre) continue;   // no room: the leader kernel looks its blocks up
        uint32_t m = ld.n;
        for (uint32_t k0 = 0; k0 < ld.n; k0 += kWave) {
            const uint32_t k = k0 + lane;
            uint32_t hk = kNoHolder;
            if (k < ld.n) {
                hk = holder_lane(t, hashes[ld.a + k]);
                hv[ld.hoff + k] = hk;
            }
            const uint64_t none = __ballot(k < ld.n && hk == kNoHolder);
            if (none) {
                m = k0 + (uint32_t)__builtin_ctzll(none);
                break;
            }
        }
        if (lane == 0) lead[slot].m = m;
    }
}

// The scoring record of a request from its prefill row and length and its
// scan element (leader slot, L*).
__device__ inline Hot make_hot(Pre pr, uint64_t e, uint32_t bt, uint32_t lstride, uint32_t zrow) {
    const uint32_t ls = (uint32_t)e, slot = (uint32_t)(e >> 32);
    const bool own = slot == kLeadOver || pr.len >= kExactTok;
    Hot o;
    o.row = pr.row;
    o.lrow = (slot < kLeadOver && !own) ? slot * lstride : zrow;
    o.len = __float_as_uint((float)pr.len);
    // ls <= n_r, so bt * ls <= len
    o.lams = own ? __float_as_uint(-1.0f)
                 : ls == kNoCap ? __float_as_uint(__builtin_inff()) : __float_as_uint((float)(bt * ls));
    return o;
}

// Scoring-order records: position k of the prefill order holds hash-order
// position pord[k], whose record takes its leader row and B_tok * L* from
// the scan (lstride: bytes per leader row; zrow: byte offset of the
// all-zero row).  A request whose leader did not fit the leader table, or
// of 2^24 tokens or more, is marked to be matched on its own.  Positions
// past the batch (kHotPad of them) get a record that the scoring kernel
// may read ahead but never scores (row 0, no leader).  With hotr, each
// request's record is also written at its index in the batch (the ranking
// sweep reads records in batch order).
__global__ __launch_bounds__(256) void assemble_kernel(uint32_t n_req, uint32_t bt, uint32_t lstride, uint32_t zrow,
                                                       const uint32_t *__restrict__ pord,
                                                       const uint64_t *__restrict__ seg,
                                                       const uint64_t *__restrict__ tpre,
                                                       const Pre *__restrict__ hrec, const Cold *__restrict__ crec,
                                                       Hot *__restrict__ hot, Cold *__restrict__ cold,
                                                       Hot *__restrict__ hotr) {
    const uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= (uint64_t)n_req + kHotPad) return;
    if (k >= n_req) {
        hot[k] = Hot{0, zrow, 0, 0};
        return;
    }
    const uint32_t i = pord[k];
    const Hot rec = make_hot(hrec[i], scanned_at(seg, tpre, i), bt, lstride, zrow);
    const Cold c = crec[i];
    hot[k] = rec;
    cold[k] = c;
    if (hotr) hotr[c.r] = rec;
}

// ---------------------------------------------------------------- batch sorts
//
// Stable LSD radix sort for the batch orders (batches of kSortMinN + 1 to
// kSortMaxN): tiles of TILE positions (sort_tile: 1,024 up to
// kSortSmallTileN positions, so that a batch of a few hundred thousand
// still spreads over every CU, else 4,096, whose digits leave in longer
// runs), one workgroup each, in passes of at most kSortMaxBits digit bits.
// A pass takes three kernels:
// sort_count_kernel counts each tile's digits into cnt[tile][digit];
// sort_colscan_kernel turns every digit's column into exclusive offsets
// over the tiles (in place) and writes the digit totals;
// sort_scatter_kernel ranks the tile's elements (each wavefront a quarter
// of the tile, 64 at a time, equal digits ranked by lane masks), stages
// them in LDS in output order and writes them out in that order, so that
// the elements of one digit leave as a contiguous run.  Equal keys keep
// their order (stable), which the prefill order relies on.
constexpr uint32_t kSortTile = 4096;           // the large tile
constexpr uint32_t kSortSmallTile = 1024;      // the small tile
constexpr uint64_t kSortSmallTileN = 1ull << 19;   // largest batch sorted in small tiles (512 of them)
constexpr uint32_t kSortMaxBits = 11;   // widest pass: the prefill order of up to 2,047 prefills in one
constexpr uint32_t kSortMaxBins = 1u << kSortMaxBits;
constexpr uint32_t kSortPassBits = 8;   // passes of the hash order and the general pair sort (faster per bit)
constexpr uint32_t kSortBinsPer = kSortMaxBins / kBlock;   // digits per thread at the widest pass
constexpr uint32_t kPrefillMaxBits = 16;   // prefill keys of more bits: rocPRIM's sort and a gather
constexpr uint64_t kSortMaxN = 1ull << 24;
constexpr uint64_t kSortMinN = 1ull << 16;   // smaller batches: rocPRIM (fewer launches)
constexpr uint64_t kForkMinN = 1ull << 16;   // batches from which a selection forks its second stream
static_assert(kSortBinsPer * kBlock == kSortMaxBins, "digits split evenly over the threads");

// Tile size of the batch sorts for n positions.
inline uint32_t sort_tile(uint64_t n) { return n <= kSortSmallTileN ? kSortSmallTile : kSortTile; }

template <uint32_t TILE>
__global__ __launch_bounds__(kBlock) void sort_count_kernel(const uint32_t *__restrict__ keys, uint32_t n,
                                                            uint32_t shift, uint32_t bits,
                                                            uint32_t *__restrict__ cnt) {
    constexpr uint32_t kPer = TILE / kBlock;   // positions per thread
    __shared__ uint32_t h[kSortMaxBins];
    const uint32_t bins = 1u << bits, mask = bins - 1;
    const uint32_t tid = threadIdx.x;
    for (uint32_t b = tid; b < bins; b += kBlock) h[b] = 0;
    __syncthreads();
    const uint64_t e0 = (uint64_t)blockIdx.x * TILE + tid;
    uint32_t kr[kPer];   // the thread's keys, all loads issued first
#pragma unroll
    for (uint32_t x = 0; x < kPer; ++x) {
        const uint64_t e = e0 + (uint64_t)x * kBlock;
        kr[x] = e < n ? keys[e] : 0u;
    }
#pragma unroll
    for (uint32_t x = 0; x < kPer; ++x)
        if (e0 + (uint64_t)x * kBlock < n) atomicAdd(h + ((kr[x] >> shift) & mask), 1u);
    __syncthreads();
    for (uint32_t b = tid; b < bins; b += kBlock) cnt[(uint64_t)blockIdx.x * bins + b] = h[b];
}

// Inclusive prefix sum over the 64 lanes of a wavefront.
__device__ inline uint32_t wave_incl_scan(uint32_t v) {
    const uint32_t lane = threadIdx.x % kWave;
#pragma unroll
    for (uint32_t off = 1; off < (uint32_t)kWave; off <<= 1) {
        const uint32_t u = __shfl_up(v, off, kWave);
        if (lane >= off) v += u;
    }
    return v;
}

// One workgroup per digit: the exclusive offsets of the digit's column
// over the tiles (in place) and the digit total.  Thread t takes kColPer
// consecutive tiles (fewer at the end), sums them, and the workgroup scans
// the sums.
constexpr uint32_t kColPer = (uint32_t)(kSortMaxN / kSortTile / kBlock);
static_assert(kColPer * kBlock * kSortTile == kSortMaxN, "column scan covers the largest batch");
static_assert(kSortSmallTileN / kSortSmallTile <= (uint64_t)kColPer * kBlock, "and the most small tiles");
__global__ __launch_bounds__(kBlock) void sort_colscan_kernel(uint32_t *__restrict__ cnt, uint32_t ntile,
                                                              uint32_t bits, uint32_t *__restrict__ tot) {
    __shared__ uint32_t wsum[kWavesPerBlock];
    const uint32_t bins = 1u << bits, b = blockIdx.x, t = threadIdx.x;
    const uint32_t per = (ntile + kBlock - 1) / kBlock;   // <= kColPer
    const uint32_t t0 = t * per;
    uint32_t c[kColPer];
    uint32_t sum = 0;
#pragma unroll
    for (uint32_t u = 0; u < kColPer; ++u) {
        c[u] = (u < per && t0 + u < ntile) ? cnt[(uint64_t)(t0 + u) * bins + b] : 0u;
        sum += c[u];
    }
    const uint32_t incl = wave_incl_scan(sum);
    if (t % kWave == kWave - 1) wsum[t / kWave] = incl;
    __syncthreads();
    uint32_t run = incl - sum;
    for (uint32_t q = 0; q < t / kWave; ++q) run += wsum[q];
#pragma unroll
    for (uint32_t u = 0; u < kColPer; ++u) {
        if (u < per && t0 + u < ntile) cnt[(uint64_t)(t0 + u) * bins + b] = run;
        run += c[u];
    }
    if (t == kBlock - 1) tot[b] = run;
}

// Exclusive prefix sum of v[0, bins) in LDS, in place, by the whole
// workgroup: thread t takes consecutive digits t*per .. t*per + per - 1
// (per = bins / kBlock, at least 1), the wavefronts scan the threads' sums
// with lane shuffles, then the four wavefront totals are added.
__device__ inline void lds_exclusive_scan(uint32_t *v, uint32_t bins) {
    __shared__ uint32_t wsum[kWavesPerBlock];
    const uint32_t t = threadIdx.x;
    const uint32_t per = bins > (uint32_t)kBlock ? bins / kBlock : 1u;
    const uint32_t b0 = t * per;
    uint32_t loc[kSortBinsPer];
    uint32_t sum = 0;
#pragma unroll
    for (uint32_t u = 0; u < kSortBinsPer; ++u) {
        loc[u] = (u < per && b0 + u < bins) ? v[b0 + u] : 0u;
        sum += loc[u];
    }
    const uint32_t incl = wave_incl_scan(sum);
    if (t % kWave == kWave - 1) wsum[t / kWave] = incl;
    __syncthreads();
    uint32_t run = incl - sum;
    for (uint32_t q = 0; q < t / kWave; ++q) run += wsum[q];
#pragma unroll
    for (uint32_t u = 0; u < kSortBinsPer; ++u) {
        if (u < per && b0 + u < bins) v[b0 + u] = run;
        run += loc[u];
    }
    __syncthreads();
}

// Lanes of the calling wavefront in `valid` whose digit equals this lane's
// (the digit's bits compared one ballot at a time).
__device__ inline uint64_t digit_peers(uint32_t d, uint32_t bits, uint64_t valid) {
    uint64_t m = valid;
    for (uint32_t j = 0; j < bits; ++j) {
        const bool bit = (d >> j) & 1u;
        const uint64_t b = __builtin_amdgcn_ballot_w64(bit);
        m &= bit ? b : ~b;
    }
    return m;
}

// Scatter of one pass.  The values are vin's, or the input positions when
// vin is null.  ASSEMBLE: the values are hash-order positions and each
// element writes its scoring records (from hrec, the scan and crec at that
// position) at its output position (and, with hotr, at the request's index
// in the batch); the kHotPad records past the batch are written too.
// Otherwise (key, value) pairs go to kout / vout.
template <bool ASSEMBLE, uint32_t TILE>
__global__ __launch_bounds__(kBlock) void sort_scatter_kernel(const uint32_t *__restrict__ kin,
                                                              const uint32_t *__restrict__ vin, uint32_t n,
                                                              uint32_t shift, uint32_t bits,
                                                              const uint32_t *__restrict__ cnt,
                                                              const uint32_t *__restrict__ tot,
                                                              uint32_t *__restrict__ kout, uint32_t *__restrict__ vout,
                                                              const Pre *__restrict__ hrec,
                                                              const uint64_t *__restrict__ seg,
                                                              const uint64_t *__restrict__ tpre,
                                                              const Cold *__restrict__ crec, uint32_t bt,
                                                              uint32_t lstride, uint32_t zrow, Hot *__restrict__ hot,
                                                              Cold *__restrict__ cold, Hot *__restrict__ hotr) {
    constexpr uint32_t kPer = TILE / kBlock;                  // positions per thread
    constexpr uint32_t kQuarter = TILE / kWavesPerBlock;      // positions per wavefront
    constexpr uint32_t kSteps = kQuarter / kWave;             // 64-position steps of a wavefront
    __shared__ uint32_t bb[kSortMaxBins];                     // the tile's first output position per digit
    __shared__ uint32_t hist[kWavesPerBlock][kSortMaxBins];   // per-wavefront counts, then their prefixes
    __shared__ uint32_t toff[kSortMaxBins];                   // first staging slot per digit
    __shared__ uint32_t sk[TILE], sv[TILE];                   // keys and values in output order
    const uint32_t bins = 1u << bits, mask = bins - 1;
    const uint32_t tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
    const uint64_t t0 = (uint64_t)blockIdx.x * TILE;
    for (uint32_t b = tid; b < bins; b += kBlock) bb[b] = tot[b];
    for (uint32_t b = lane; b < bins; b += kWave) hist[w][b] = 0;
    __syncthreads();
    lds_exclusive_scan(bb, bins);   // the digits' first output positions
    for (uint32_t b = tid; b < bins; b += kBlock) bb[b] += cnt[(uint64_t)blockIdx.x * bins + b];
    if (ASSEMBLE && blockIdx.x == 0 && tid < kHotPad) hot[(uint64_t)n + tid] = Hot{0, zrow, 0, 0};
    // this wavefront's quarter of the tile: keys and values, loads first
    const uint64_t e0 = t0 + (uint64_t)w * kQuarter + lane;
    uint32_t kr[kSteps], vr[kSteps], rk[kSteps];
#pragma unroll
    for (uint32_t x = 0; x < kSteps; ++x) {
        const uint64_t e = e0 + (uint64_t)x * kWave;
        kr[x] = e < n ? kin[e] : 0u;
        vr[x] = e < n ? (vin ? vin[e] : (uint32_t)e) : 0u;
    }
    __syncthreads();
    // rank within the wavefront's quarter, step by step
#pragma unroll
    for (uint32_t x = 0; x < kSteps; ++x) {
        const bool valid = e0 + (uint64_t)x * kWave < n;
        const uint32_t d = (kr[x] >> shift) & mask;
        const uint64_t peers = digit_peers(d, bits, __builtin_amdgcn_ballot_w64(valid));
        const uint32_t at = hist[w][d];
        if (valid && lane == (uint32_t)__builtin_ctzll(peers)) hist[w][d] = at + (uint32_t)__builtin_popcountll(peers);
        rk[x] = at + __builtin_amdgcn_mbcnt_hi((uint32_t)(peers >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u));
    }
    __syncthreads();
    // per digit: the wavefronts' prefixes (in place) and the tile count
    for (uint32_t b = tid; b < bins; b += kBlock) {
        uint32_t run = 0;
#pragma unroll
        for (uint32_t q = 0; q < kWavesPerBlock; ++q) {
            const uint32_t c = hist[q][b];
            hist[q][b] = run;
            run += c;
        }
        toff[b] = run;
    }
    __syncthreads();
    lds_exclusive_scan(toff, bins);   // the digits' first staging slots
    // stage in output order
#pragma unroll
    for (uint32_t x = 0; x < kSteps; ++x) {
        if (e0 + (uint64_t)x * kWave < n) {
            const uint32_t d = (kr[x] >> shift) & mask;
            const uint32_t pos = toff[d] + hist[w][d] + rk[x];
            sk[pos] = kr[x];
            sv[pos] = vr[x];
        }
    }
    __syncthreads();
    // write out in output order: one digit's elements are consecutive
    const uint32_t nt = n - t0 < (uint64_t)TILE ? (uint32_t)(n - t0) : TILE;
#pragma unroll
    for (uint32_t x = 0; x < kPer; ++x) {
        const uint32_t j = x * kBlock + tid;
        if (j < nt) {
            const uint32_t k = sk[j];
            const uint32_t d = (k >> shift) & mask;
            const uint32_t o = bb[d] + (j - toff[d]);
            if (ASSEMBLE) {
                const uint32_t e = sv[j];
                const Hot rec = make_hot(hrec[e], scanned_at(seg, tpre, e), bt, lstride, zrow);
                const Cold c = crec[e];
                hot[o] = rec;
                cold[o] = c;
                if (hotr) hotr[c.r] = rec;
            } else {
                kout[o] = k;
                vout[o] = sv[j];
            }
        }
    }
}

// Read-only data that is uniform across a wavefront (request records, hash
// runs) is read through the constant address space, which the compiler
// serves with scalar loads into SGPRs.
template <typename T>
using cptr = const __attribute__((address_space(4))) T *;

template <typename T>
__device__ inline cptr<T> as_const(const T *p) {
    return (cptr<T>)(const __attribute__((address_space(4))) void *)(uintptr_t)p;
}

__device__ inline Hot load_hot(const Hot *base, uint32_t i) {
    const cptr<uint32_t> w = as_const((const uint32_t *)(base + i));
    Hot x;
    x.row = w[0];
    x.lrow = w[1];
    x.len = w[2];
    x.lams = w[3];
    return x;
}

__device__ inline Cold load_cold(const Cold *base, uint32_t i) {
    return Cold{as_const((const uint32_t *)base)[i]};
}

// Lane masks of a wavefront: ballot turns a per-lane predicate into a
// uniform 64-bit mask (held in scalar registers), in_mask reads a lane's
// bit back as a predicate.  Per-column "alive" and "need" sets are kept as
// masks so that their tests and combinations are scalar operations.
using lmask = uint64_t;

__device__ inline lmask ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
__device__ inline bool in_mask(lmask m) { return __builtin_amdgcn_inverse_ballot_w64(m); }

// v_writelane: lane `l` (uniform) of `old` takes the uniform value `v`, the
// other lanes keep theirs.  The compiler offers no builtin for it, so the
// intrinsic is declared by its name.
extern "C" __device__ int amdgcn_writelane(int v, int l, int old) __asm("llvm.amdgcn.writelane.i32");
__device__ inline uint32_t write_lane(uint32_t v, uint32_t l, uint32_t old) {
    return (uint32_t)amdgcn_writelane((int)v, (int)l, (int)old);
}

// Holder value of a hash that is the same on every lane (scalar loads of
// both candidate buckets' keys and values).
__device__ inline uint32_t holder_uniform(const Table &t, uint64_t h) {
    uint32_t b1, b2;
    buckets_of(h, t.shift, b1, b2);
    const cptr<uint64_t> k = as_const(t.keys);
    const cptr<uint32_t> v = as_const(t.vals);
    const uint64_t k10 = k[2 * (uint64_t)b1], k11 = k[2 * (uint64_t)b1 + 1];
    const uint64_t k20 = k[2 * (uint64_t)b2], k21 = k[2 * (uint64_t)b2 + 1];
    const uint32_t v10 = v[2 * (uint64_t)b1], v11 = v[2 * (uint64_t)b1 + 1];
    const uint32_t v20 = v[2 * (uint64_t)b2], v21 = v[2 * (uint64_t)b2 + 1];
    if (h == 0) return kNoHolder;
    return k10 == h ? v10 : k11 == h ? v11 : k20 == h ? v20 : k21 == h ? v21 : kNoHolder;
}

// Lane masks of the holders of a (uniform) holder value on the C columns of
// the wavefront whose first decode is `base` (a multiple of 64 * C): the
// wavefront's words of the bitmap row (always loaded, from row 0 when the
// value is not a row, so that the load does not wait on a branch), or the
// one lane of a single holder, or none.
template <int C>
__device__ inline void holder_masks(const Table &t, uint32_t v, uint32_t base, lmask (&m)[C]) {
    const bool row = v < kHeldOne;
    const cptr<uint64_t> w = as_const(t.bits + (uint64_t)(row ? v : 0u) * t.bpitch + base / kWave);
    const uint32_t d = v & ~kHeldOne;
#pragma unroll
    for (int q = 0; q < C; ++q) {
        const uint32_t o = d - (base + (uint32_t)q * kWave);
        const lmask one = (v != kNoHolder && o < (uint32_t)kWave) ? (1ull << o) : 0ull;
        m[q] = row ? w[q] : one;
    }
}

// First-miss scan of one request's run on the columns in alive[] (the
// columns that need it), starting at block `start` (uniform, < n) whose
// holder value v0 was looked up beforehand.  Past the first block, W blocks
// are looked up per step, their holder lookups issued together.  lam[]
// holds bt * start on entry for those columns and bt * (first-miss index)
// on return (bt = tokens per block).
template <int W, int C>
__device__ inline void probe_from(const Table &t, uint32_t base, cptr<uint64_t> run, uint32_t n, uint32_t start,
                                  lmask (&alive)[C], uint32_t (&lam)[C], uint32_t bt, uint32_t v0) {
    lmask m[C];
    holder_masks<C>(t, v0, base, m);
#pragma unroll
    for (int q = 0; q < C; ++q) {
        alive[q] &= m[q];
        lam[q] += in_mask(alive[q]) ? bt : 0u;
    }
    for (uint32_t i0 = start + 1; i0 < n; i0 += W) {
        lmask any = 0;
#pragma unroll
        for (int q = 0; q < C; ++q) any |= alive[q];
        if (!any) break;
        uint32_t v[W];
#pragma unroll
        for (int w = 0; w < W; ++w) v[w] = i0 + w < n ? holder_uniform(t, run[i0 + w]) : kNoHolder;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            if (i0 + w >= n) break;
            holder_masks<C>(t, v[w], base, m);
#pragma unroll
            for (int q = 0; q < C; ++q) {
                alive[q] &= m[q];
                lam[q] += in_mask(alive[q]) ? bt : 0u;
            }
        }
    }
}

// Prefix lengths of every leader on every decode: one wavefront per
// (leader, kLeadGroups groups of 64 decodes), looping over such tasks (the
// leader count is read from device memory, so every wavefront ends after at
// most ceil(tasks / wavefronts) of them).  A task takes the leader's blocks
// 64 at a time, lane k block k: its holder value (looked up by
// lead_holder_kernel, or here when there was no room), then, per group, the
// word of its bitmap row over the group's 64 decodes (or the one-hot word of
// a single holder).  An inclusive AND across lanes, seeded with the group's
// decodes still matching, gives in lane k the decodes that hold every block
// up to k; it only loses bits as k grows, so decode l matches exactly the
// blocks below the first lane whose word lacks bit l, found by binary
// search over the words in LDS.  Writes B_tok * j for the task's decodes,
// in fp32 (exact below 2^24; only requests shorter than that read it,
// capped by their own length).
// Inclusive AND over lanes 0..l of a 32-bit value, in lane l, with DPP:
// shifts right by 1, 2, 4 and 8 within each row of 16 lanes (a lane with
// no source takes all ones), then the last lane of row 0 into row 1 and of
// row 2 into row 3, then the last lane of row 1 into rows 2 and 3.  Every
// lane must be active.
__device__ inline uint32_t wave_and_prefix_u32(uint32_t v) {
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x111, 0xF, 0xF, false);   // row_shr 1
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x112, 0xF, 0xF, false);   // row_shr 2
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x114, 0xF, 0xF, false);   // row_shr 4
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x118, 0xF, 0xF, false);   // row_shr 8
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x142, 0xA, 0xF, false);   // row_bcast 15
    v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x143, 0xC, 0xF, false);   // row_bcast 31
    return v;
}

__device__ inline uint64_t wave_and_prefix_u64(uint64_t v) {
    const uint32_t lo = wave_and_prefix_u32((uint32_t)v), hi = wave_and_prefix_u32((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Groups of 64 decodes per task: the task's groups share each block's
// holder value (and its load); their bitmap words load side by side.
constexpr uint32_t kLeadGroups = 2;

__global__ __launch_bounds__(kBlock) void lead_kernel(Table t, uint32_t D, uint32_t bt, const Lead *__restrict__ lead,
                                                      const unsigned int *__restrict__ n_lead, uint32_t lead_cap,
                                                      const uint32_t *__restrict__ hv,
                                                      const uint64_t *__restrict__ hashes, uint32_t ngroup,
                                                      float *__restrict__ lam_out) {
    __shared__ uint64_t pw[kWavesPerBlock][kLeadGroups][kWave];
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t wv = wave_index();
    const uint32_t nl_all = *n_lead;
    const uint32_t nl = nl_all < lead_cap ? nl_all : lead_cap;
    const uint32_t ntg = (ngroup + kLeadGroups - 1) / kLeadGroups;   // tasks per leader
    const uint64_t tasks = (uint64_t)nl * ntg;
    const uint64_t nw = (uint64_t)gridDim.x * kWavesPerBlock;
    for (uint64_t task = (uint64_t)blockIdx.x * kWavesPerBlock + wv; task < tasks; task += nw) {
        const uint32_t slot = (uint32_t)(task / ntg), g0 = (uint32_t)(task % ntg) * kLeadGroups;
        const cptr<uint32_t> w = as_const((const uint32_t *)(lead + slot));
        const uint64_t a = ((uint64_t)w[1] << 32) | (uint64_t)w[0];
        const uint64_t hoff = ((uint64_t)w[3] << 32) | (uint64_t)w[2];
        const uint32_t n = w[4], m = w[5];
        const bool pre = m != kNoPre;
        const uint32_t nb = pre ? m : n;   // blocks to take (held by someone before block m)
        // per group: the decodes (lanes) holding every block so far, and
        // this lane's decode's leading blocks held; a group past the pool
        // holds none
        uint64_t alive[kLeadGroups];
        uint32_t j[kLeadGroups];
#pragma unroll
        for (uint32_t q = 0; q < kLeadGroups; ++q) {
            alive[q] = g0 + q < ngroup ? ~0ull : 0ull;
            j[q] = 0;
        }
        auto live = [&]() {
            uint64_t x = 0;
#pragma unroll
            for (uint32_t q = 0; q < kLeadGroups; ++q) x |= alive[q];
            return x != 0;
        };
        for (uint32_t k0 = 0; k0 < nb && live(); k0 += kWave) {
            const uint32_t k = k0 + lane;
            const uint32_t nk = nb - k0 < (uint32_t)kWave ? nb - k0 : (uint32_t)kWave;
            uint32_t v = kNoHolder;
            if (k < nb) v = pre ? hv[hoff + k] : holder_lane(t, hashes[a + k]);
#pragma unroll
            for (uint32_t q = 0; q < kLeadGroups; ++q) {
                const uint32_t g = g0 + q;
                uint64_t word = 0;
                if (g < ngroup) {
                    if (v < kHeldOne) {
                        word = t.bits[(uint64_t)v * t.bpitch + g];
                    } else if (v != kNoHolder) {
                        const uint32_t o = (v & ~kHeldOne) - g * kWave;
                        word = o < (uint32_t)kWave ? 1ull << o : 0ull;
                    }
                }
                pw[wv][q][lane] = wave_and_prefix_u64(word & alive[q]);
            }
            __builtin_amdgcn_wave_barrier();
            // lane l: the number of leading words (of nk) holding bit l
#pragma unroll
            for (uint32_t q = 0; q < kLeadGroups; ++q) {
                uint32_t lo = 0, hi = nk;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) / 2;
                    if ((pw[wv][q][mid] >> lane) & 1ull) lo = mid + 1;
                    else hi = mid;
                }
                j[q] += lo;
                alive[q] = pw[wv][q][nk - 1];
            }
            __builtin_amdgcn_wave_barrier();
        }
#pragma unroll
        for (uint32_t q = 0; q < kLeadGroups; ++q) {
            const uint32_t d = (g0 + q) * kWave + lane;
            if (g0 + q < ngroup && d < D) lam_out[(uint64_t)slot * D + d] = (float)(bt * j[q]);
        }
    }
}

// Buffer-resource word 3 for raw (untyped, unswizzled) buffer access on gfx9-class targets.
constexpr int kBufferFlags = 0x00020000;

__device__ inline float2 load_row(__amdgpu_buffer_rsrc_t r, uint32_t lane_off, uint32_t row_off) {
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)lane_off, (int)row_off, 0));
}

__device__ inline uint32_t load_lam(__amdgpu_buffer_rsrc_t r, uint32_t lane_off, uint32_t row_off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)lane_off, (int)row_off, 0);
}

// One wavefront per (run of scoring-order requests, group of 64*C decodes);
// lane l holds decodes g*64*C + q*64 + l, q < C.  For each request of the
// run: prefix lengths min(leader's, L*), non-cached tokens, feasibility and
// cost (Eqs. (2)-(7)), then the group's K best feasible (score, index) keys
// into partial[group][position][0..K).  Token counts are below 2^24 here,
// so x = l - lambda and the feasibility test x <= xm_d are exact in fp32
// and give the costs of integer arithmetic; a request no longer than every
// limit xm_d of the group is feasible on all of them and skips the test.
// A request marked in its record (its leader did not fit the leader table,
// or it has 2^24 tokens or more) is matched from block 0 on its own and
// scored in integers.  Requests of one prefill are consecutive, so the
// snapshot row stays in registers and is reloaded only when the prefill
// changes; the leader's prefix lengths are kept too, and the next
// request's are fetched during the current step only when its leader row
// differs.  Records are read two requests ahead.  Requests are taken in
// chunks of 64/K whose keys are gathered one per lane and stored together.
// The cost of a pair with x non-cached tokens from its derived row(s), as
// fp32 bits: the direct route, or the cheaper of the direct and the staged
// route (costs are non-negative, so the smaller bits are the smaller cost;
// ties keep the direct route's value, which is the same).
template <bool TWO>
__device__ inline uint32_t route_cost(float x, float2 r1, float2 r2) {
    const uint32_t c1 = __float_as_uint(fmaf(x, r1.x, r1.y));
    if (!TWO) return c1;
    return min(c1, __float_as_uint(fmaf(x, r2.x, r2.y)));
}

// Merged mode (MERGE, at most kMaxMergeGroups groups; used for a pool of
// one group, where it saves the merge kernel): a workgroup is one run,
// its wavefront w the decode group w; at the end of each chunk of requests
// the wavefronts put their top-k keys in LDS (two buffers, alternating by
// chunk), and after one barrier each wavefront merges a share of the
// chunk's requests over all groups and writes their outputs.  A buffer is
// written again only two chunks later, after the next barrier, which every
// wavefront reaches only once its merge of the buffer is done.  Workgroups
// go to the XCDs in turn, and XCD x takes the x-th contiguous eighth of the
// runs, so its L2 holds the snapshot rows of its own prefills.
constexpr uint32_t kMaxMergeGroups = 8;

// Without per-pair outputs the kernel is held to 80 registers, so that a
// SIMD keeps 6 wavefronts (the staged-route variant needs one register
// more than that when left alone).
template <int K, int W, int C, bool PAIRS, bool TWO, bool MERGE>
__global__ __launch_bounds__(MERGE ? kWave * kMaxMergeGroups : kBlock, PAIRS ? 1 : 6)
void score_kernel(Snap s, Table t, const Hot *__restrict__ hot, const Cold *__restrict__ cold,
                  const float *__restrict__ lead_lam, uint32_t lead_rows, const uint64_t *__restrict__ hashes,
                  const uint32_t *__restrict__ len_tokens, const uint64_t *__restrict__ hash_off,
                  const uint32_t *__restrict__ n_valid, uint32_t n_req, uint32_t run_len, uint32_t n_runs,
                  uint32_t ngroup, uint64_t *__restrict__ partial, PairOut po, uint32_t k_out,
                  int32_t *__restrict__ out_idx, float *__restrict__ out_score) {
    __shared__ uint64_t mkeys[MERGE ? 2 : 1][MERGE ? kMaxMergeGroups : 1][kWave];
    const uint32_t lane = threadIdx.x % kWave;
    uint32_t run, grp;
    if (MERGE) {
        const uint32_t rpx = (n_runs + kXcds - 1) / kXcds;
        run = (blockIdx.x % kXcds) * rpx + blockIdx.x / kXcds;
        grp = wave_index();
    } else if (ngroup % kXcds == 0) {
        // workgroups go to the XCDs in turn: XCD x takes groups
        // [x*gx, (x+1)*gx), so its decodes' snapshot columns stay in its
        // own L2; the waves of a workgroup take consecutive runs of one group
        const uint32_t gx = ngroup / kXcds, x = blockIdx.x % kXcds, k = blockIdx.x / kXcds;
        grp = x * gx + k % gx;
        run = (k / gx) * kWavesPerBlock + wave_index();
    } else {
        const uint32_t gw = blockIdx.x * kWavesPerBlock + wave_index();
        run = gw / ngroup;
        grp = gw % ngroup;
    }
    if (run >= n_runs) return;
    const uint32_t nv = *n_valid;
    const uint32_t i0 = run * run_len;
    if (i0 >= nv) return;
    const uint32_t i1 = (i0 + run_len < nv) ? i0 + run_len : nv;
    const uint32_t base = grp * (kWave * C);
    const uint32_t bt = s.block_tokens;
    uint32_t d[C];
    float xmf[C];
    bool act[C];
    // x = l - lambda is feasible iff x < xlim, i.e. x <= xlim - 1 for
    // xlim >= 1; xlim = 0 never is (limit -1).  Limits above 2^24 are taken
    // as 2^24, which every x scored in fp32 is below.  A column past the
    // pool has limit NaN, which no x passes, whatever its loads read.  xlo:
    // the least limit of the lane's decodes as fp32 bits, 0 when one is
    // never feasible (so a group with columns past the pool, and requests
    // of at least one token, never take the all-feasible path).
    uint32_t xlo = 0xFFFFFFFFu;
#pragma unroll
    for (int q = 0; q < C; ++q) {
        d[q] = base + q * kWave + lane;
        act[q] = d[q] < s.D;
        const uint64_t xlim = act[q] ? s.dxlim[d[q]] : 0;
        xmf[q] = !act[q] ? __builtin_nanf("")
                 : xlim == 0 ? -1.0f
                             : (float)(xlim - 1 < kExactTok ? xlim - 1 : (uint64_t)kExactTok);
        xlo = min(xlo, xlim == 0 ? 0u : __float_as_uint(xmf[q]));
    }
    // column q of the lane is at lane offset (base + lane + 64 q) * size;
    // the 64 q part is a constant that the loads carry in their offset
    // field, so the lane needs one offset register per table.  Columns past
    // the pool read what follows the last decode: the next row, or the
    // kRowPad elements allocated after the last row.
    constexpr uint32_t kRowStep = kWave * (uint32_t)sizeof(float2), kLamStep = kWave * (uint32_t)sizeof(float);
    const uint32_t voff = (base + lane) * (uint32_t)sizeof(float2);
    const uint32_t loff = (base + lane) * (uint32_t)sizeof(float);
    // a request of at most xall tokens (fp32 bits) is feasible on every
    // decode of the group
    const uint32_t xall = wave_min_u32_dpp(xlo);
    const cptr<uint64_t> chash = as_const(hashes);
    // rows of (seconds per token, constant part) and the leaders' prefix
    // lengths through buffer resources: a row's byte offset is the scalar
    // offset, the column's the lane offset
    const uint64_t sl_bytes = ((uint64_t)s.P * s.slp + kRowPad) * sizeof(float2);   // < 2^32 (checked at load)
    const uint64_t ll_bytes = ((uint64_t)lead_rows * s.D + kRowPad) * sizeof(float);   // < 2^32 (capped)
    const __amdgpu_buffer_rsrc_t slr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)s.sl, (short)0, (int)(uint32_t)(sl_bytes < 0xFFFFFFFFull ? sl_bytes : 0xFFFFFFFFull), kBufferFlags);
    const __amdgpu_buffer_rsrc_t llr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)lead_lam, (short)0, (int)(uint32_t)(ll_bytes < 0xFFFFFFFFull ? ll_bytes : 0xFFFFFFFFull),
        kBufferFlags);
    const __amdgpu_buffer_rsrc_t srr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(TWO ? s.sr : s.sl), (short)0,
        (int)(uint32_t)(sl_bytes < 0xFFFFFFFFull ? sl_bytes : 0xFFFFFFFFull), kBufferFlags);
    Hot c0 = load_hot(hot, i0);
    Hot c1 = load_hot(hot, i0 + 1);
    float2 rowv[C], rowv2[C];   // the current prefill's row (and its staged-route row)
    uint32_t rowcur = c0.row;
    // the current leader's B_tok * j (the next one's while it loads), as
    // fp32 bits: non-negative, so their order is that of the unsigned bits
    uint32_t laml[C];
#pragma unroll
    for (int q = 0; q < C; ++q) {
        rowv[q] = load_row(slr, voff + q * kRowStep, c0.row);
        rowv2[q] = TWO ? load_row(srr, voff + q * kRowStep, c0.row) : rowv[q];
        laml[q] = load_lam(llr, loff + q * kLamStep, c0.lrow);
    }
    constexpr uint32_t kPer = kWave / K;   // requests whose keys one store writes
    uint32_t pc_bits = 0xFFFFFFFFu, pc_idx = 0xFFFFFFFFu;   // gathered keys (empty = ~0)

    // one request's column costs (fp32 bits, ~0 where infeasible):
    // scoring-order position i, its record and the next one's (whose leader
    // values are fetched while i is scored)
    auto cost = [&](uint32_t i, const Hot &cur, const Hot &nxt, Hot &ahead, uint32_t (&cb)[C]) {
        // the lane offsets of the loads below are tied to the request (an
        // empty asm, no instruction) so that each column's offset stays in
        // the load's offset field instead of a register of its own
        if (cur.row != rowcur) {
            uint32_t vo = voff;
            asm("" : "+v"(vo) : "s"(i));
#pragma unroll
            for (int q = 0; q < C; ++q) {
                rowv[q] = load_row(slr, vo + q * kRowStep, cur.row);
                if (TWO) rowv2[q] = load_row(srr, vo + q * kRowStep, cur.row);
            }
            rowcur = cur.row;
        }
        // the record two ahead, issued after the last use of the loaded
        // records' fields (scalar loads complete out of order, so a use
        // after it would wait for it)
        __builtin_amdgcn_sched_barrier(0);
        ahead = load_hot(hot, i + 2);
        uint32_t r_out = 0;
        if (PAIRS) r_out = load_cold(cold, i).r;
        // this request's prefix lengths B_tok * j (fp32 bits): its leader's,
        // capped by its own common run with the leader; then the next
        // request's leader values, if its leader row differs, are loaded
        // over the current ones, whose last use this is (with staged routes,
        // after the costs: there the kernel has no registers for both sets
        // beside the costs' operands)
        uint32_t lam[C];
#pragma unroll
        for (int q = 0; q < C; ++q) lam[q] = min(laml[q], cur.lams);
        auto reload = [&]() {
            if (nxt.lrow != cur.lrow) {
                uint32_t lo = loff;
                asm("" : "+v"(lo) : "s"(i));
#pragma unroll
                for (int q = 0; q < C; ++q) laml[q] = load_lam(llr, lo + q * kLamStep, nxt.lrow);
            }
        };
        if (!TWO) reload();
        if ((int32_t)cur.lams < 0) {
            // matched on its own from block 0, in integers (exact)
            const uint32_t r = load_cold(cold, i).r;
            const uint32_t len = as_const(len_tokens)[r];
            const uint64_t ha = as_const(hash_off)[r];
            const uint32_t hn = (uint32_t)(as_const(hash_off)[r + 1] - ha);
            lmask alive[C];
            uint32_t lam[C];
#pragma unroll
            for (int q = 0; q < C; ++q) {
                lam[q] = 0;
                alive[q] = ~0ull;
            }
            if (hn)
                probe_from<W, C>(t, base, chash + ha, hn, 0, alive, lam, bt, holder_uniform(t, chash[ha]));
#pragma unroll
            for (int q = 0; q < C; ++q) {
                const uint32_t x = len - lam[q];
                const uint64_t xlim = act[q] ? s.dxlim[d[q]] : 0;
                const bool feas = (uint64_t)x < xlim;
                const float cost = __uint_as_float(route_cost<TWO>((float)x, rowv[q], rowv2[q]));
                if (PAIRS && act[q]) {
                    const uint64_t o = (uint64_t)r_out * s.D + d[q];
                    const uint32_t jq = lam[q] / bt;
                    if (po.j) po.j[o] = (uint16_t)(jq < 0xFFFFu ? jq : 0xFFFFu);
                    if (po.feas) po.feas[o] = feas ? 1 : 0;
                    if (po.score) po.score[o] = cost;
                }
                cb[q] = feas ? __float_as_uint(cost) : 0xFFFFFFFFu;
            }
        } else {
            // non-cached tokens (Eq. (2) / bpt), feasibility and the cost of Eq. (5)
            const float lenf = __uint_as_float(cur.len);
            if (!PAIRS && cur.len <= xall) {
#pragma unroll
                for (int q = 0; q < C; ++q)
                    cb[q] = route_cost<TWO>(lenf - __uint_as_float(lam[q]), rowv[q], rowv2[q]);
            } else {
#pragma unroll
                for (int q = 0; q < C; ++q) {
                    const float x = lenf - __uint_as_float(lam[q]);
                    const bool feas = x <= xmf[q];
                    const float cost = __uint_as_float(route_cost<TWO>(x, rowv[q], rowv2[q]));
                    if (PAIRS && act[q]) {
                        const uint64_t o = (uint64_t)r_out * s.D + d[q];
                        const uint32_t jq = (uint32_t)__uint_as_float(lam[q]) / bt;
                        if (po.j) po.j[o] = (uint16_t)(jq < 0xFFFFu ? jq : 0xFFFFu);
                        if (po.feas) po.feas[o] = feas ? 1 : 0;
                        if (po.score) po.score[o] = cost;
                    }
                    cb[q] = feas ? __float_as_uint(cost) : 0xFFFFFFFFu;
                }
            }
        }
        if (TWO) reload();
    };
    auto lane_min = [&](const uint32_t (&cb)[C]) {
        uint32_t lm = cb[0];
#pragma unroll
        for (int q = 1; q < C; ++q) lm = min(lm, cb[q]);
        return lm;
    };
    // one of the group's best, of cost bits mn (uniform; ~0 when no
    // feasible candidate is left, and nothing is kept): the least decode
    // index holding it, i.e. the lowest lane holding it in the first column
    // that holds it, whose cost is then removed; its key goes to lane e
    auto place = [&](uint32_t e, uint32_t mn, uint32_t (&cb)[C], bool more) {
        if (mn == 0xFFFFFFFFu) return false;
        uint32_t dm = 0;
#pragma unroll
        for (int q = 0; q < C; ++q) {
            const lmask m = ballot(cb[q] == mn);
            if (m) {
                const uint32_t l = (uint32_t)__builtin_ctzll(m);
                dm = base + q * kWave + l;
                if (more && lane == l) cb[q] = 0xFFFFFFFFu;
                break;
            }
        }
        pc_bits = write_lane(mn, e, pc_bits);
        pc_idx = write_lane(dm, e, pc_idx);
        return true;
    };
    // one request scored and its K best kept: least cost bits, then least
    // decode index
    auto step = [&](uint32_t i, uint32_t g0, const Hot &cur, const Hot &nxt, Hot &ahead) {
        uint32_t cb[C];
        cost(i, cur, nxt, ahead, cb);
        const uint32_t slot = i - g0;
#pragma unroll
        for (int r = 0; r < K; ++r)
            if (!place(slot * K + (uint32_t)r, wave_min_u32_dpp(lane_min(cb)), cb, r + 1 < K)) break;
    };

    for (uint32_t g0 = i0; g0 < i1; g0 += kPer) {
        const uint32_t g1 = (g0 + kPer < i1) ? g0 + kPer : i1;
        uint32_t i = g0;
        // three requests per trip: each record is loaded into the registers
        // of the one whose step has just ended, so the records rotate
        // without copies; for K = 1 the three requests' minima are taken
        // together (not with per-pair outputs or staged routes, whose
        // variants would then need more registers than 6 wavefronts per
        // SIMD leave)
        for (; i + 3 <= g1; i += 3) {
            Hot c2, c3, c4;
            if (K == 1 && !PAIRS && !TWO) {
                uint32_t ca[C], cb[C], cc[C];
                cost(i, c0, c1, c2, ca);
                cost(i + 1, c1, c2, c3, cb);
                cost(i + 2, c2, c3, c4, cc);
                uint32_t ma, mb, mc;
                wave_min3_u32(lane_min(ca), lane_min(cb), lane_min(cc), ma, mb, mc);
                place(i - g0, ma, ca, false);
                place(i + 1 - g0, mb, cb, false);
                place(i + 2 - g0, mc, cc, false);
            } else {
                step(i, g0, c0, c1, c2);
                step(i + 1, g0, c1, c2, c3);
                step(i + 2, g0, c2, c3, c4);
            }
            c0 = c3;
            c1 = c4;
        }
        for (; i < g1; ++i) {
            Hot c2;
            step(i, g0, c0, c1, c2);
            c0 = c1;
            c1 = c2;
        }
        const uint64_t key = ((uint64_t)pc_bits << 32) | (uint64_t)pc_idx;
        if (MERGE) {
            const uint32_t buf = ((g0 - i0) / kPer) & 1u;
            mkeys[buf][grp][lane] = key;
            __syncthreads();
            // request slot sl of the chunk (its keys in lanes sl*K ..
            // sl*K+K-1 of every group) is merged by lane sl / ngroup of
            // wavefront sl % ngroup
            const uint32_t sl = grp + lane * ngroup;
            if (sl < g1 - g0) {
                uint64_t best[K];
#pragma unroll
                for (int q = 0; q < K; ++q) best[q] = kEmptyKey;
                for (uint32_t g = 0; g < ngroup; ++g) {
#pragma unroll
                    for (int q = 0; q < K; ++q) {
                        const uint64_t x = mkeys[buf][g][sl * K + q];
                        if (x < best[K - 1]) topk_insert<K>(best, x);
                    }
                }
                const uint64_t o = (uint64_t)cold[g0 + sl].r * k_out;
                for (uint32_t q = 0; q < k_out; ++q) {
                    const uint64_t m = best[q];
                    out_idx[o + q] = m == kEmptyKey ? -1 : (int32_t)(uint32_t)m;
                    out_score[o + q] = m == kEmptyKey ? __builtin_inff() : __uint_as_float((uint32_t)(m >> 32));
                }
            }
        } else if (lane < (g1 - g0) * K) {
            // the lane tied to the chunk (an empty asm, no instruction), so
            // that the store's address is formed here instead of held in
            // registers through the loop
            uint32_t ln = lane;
            asm("" : "+v"(ln) : "s"(g0));
            partial[((uint64_t)grp * n_req + g0) * K + ln] = key;
        }
        pc_bits = 0xFFFFFFFFu;
        pc_idx = 0xFFFFFFFFu;
    }
}

// Merge the per-group keys of every scoring-order request into its top-k
// (ascending (score, index)) and write it at the request's own position;
// invalid requests (ordered last) get index -1 and score NaN.
template <int K>
__global__ __launch_bounds__(256) void reduce_kernel(uint32_t n_req, uint32_t nchunk, uint32_t k,
                                                     const uint64_t *__restrict__ partial,
                                                     const Cold *__restrict__ cold,
                                                     const uint32_t *__restrict__ n_valid,
                                                     int32_t *__restrict__ out_idx, float *__restrict__ out_score) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_req) return;
    const uint64_t o = (uint64_t)cold[i].r * k;
    if (i >= *n_valid) {
        for (uint32_t q = 0; q < k; ++q) {
            out_idx[o + q] = -1;
            out_score[o + q] = __builtin_nanf("");
        }
        return;
    }
    uint64_t best[K];
#pragma unroll
    for (int q = 0; q < K; ++q) best[q] = kEmptyKey;
    for (uint32_t c = 0; c < nchunk; ++c) {
        const uint64_t *src = partial + ((uint64_t)c * n_req + i) * K;
#pragma unroll
        for (int q = 0; q < K; ++q) {
            const uint64_t x = src[q];
            if (x < best[K - 1]) topk_insert<K>(best, x);
        }
    }
#pragma unroll
    for (int q = 0; q < K; ++q) {
        if ((uint32_t)q < k) {
            const uint64_t m = best[q];
            out_idx[o + q] = m == kEmptyKey ? -1 : (int32_t)(uint32_t)m;
            out_score[o + q] = m == kEmptyKey ? __builtin_inff() : __uint_as_float((uint32_t)(m >> 32));
        }
    }
}

// ---------------------------------------------------------------- ranking sweep
//
// Re-ranking of a batch under congestion scenarios (Sec. V-D).  Prefix
// lengths do not depend on congestion: every request's non-cached tokens on
// every decode come from its scoring record (leader row and cap, as in
// score_kernel) once, and only seconds per token change per scenario.
// Under scenario s the pair costs x * spt_s(p, d) + (L + load term), with
// spt_s from the scenario's congestion by the same expression as the
// snapshot's derived rows, so a scenario equal to the snapshot reproduces
// the selection bit for bit.

// Seconds per non-cached token of every (scenario, p, d).
__global__ __launch_bounds__(256) void derive_scen_kernel(Snap s, const float *__restrict__ util_scen, uint64_t n,
                                                          float *__restrict__ spt) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint64_t pd = i % ((uint64_t)s.P * s.D);
    const uint32_t p = (uint32_t)(pd / s.D);
    spt[i] = sec_per_token(s, s.tier_map[pd] & 3u, p, util_scen[i]);
}

constexpr uint32_t kSweepThreads = 256;   // requests per workgroup, one per thread, in batch order
constexpr uint32_t kSweepScen = 32;       // scenarios per workgroup
constexpr uint32_t kSweepMaxTab = 8192;   // largest P * Dp kept in LDS (two fp32 tables; three when held)
constexpr uint32_t kSweepHold = 3;        // scenario-table entries a thread holds while the previous is scored

// Ascending top-K list of fp32 cost bits (unsigned order) and decodes:
// insert (key, d) by min / median-of-three on the values and selects on the
// indices; decodes come in ascending order and only a strictly smaller key
// moves ahead, so equal costs keep the lower index first.
template <int K>
__device__ inline void topk_ins32(uint32_t (&t)[K], uint32_t (&ix)[K], uint32_t key, uint32_t d) {
    bool c[K];
#pragma unroll
    for (int q = 0; q < K; ++q) c[q] = key < t[q];
#pragma unroll
    for (int q = K - 1; q >= 1; --q) {
        ix[q] = c[q - 1] ? ix[q - 1] : (c[q] ? d : ix[q]);
        // the median of t[q-1], t[q] and key, in the form the compiler
        // turns into one median-of-three instruction
        t[q] = max(min(t[q - 1], t[q]), min(max(t[q - 1], t[q]), key));
    }
    ix[0] = c[0] ? d : ix[0];
    t[0] = min(t[0], key);
}

// Decodes db .. db+63 holding a hash with holder value v, as a bit mask
// (db a multiple of 64, or 0).
__device__ inline uint64_t held_mask(const Table &t, uint32_t v, uint32_t db) {
    if (v == kNoHolder) return 0;
    if (v & kHeldOne) {
        const uint32_t o = (v & ~kHeldOne) - db;
        return o < (uint32_t)kWave ? 1ull << o : 0ull;
    }
    return t.bits[(uint64_t)v * t.bpitch + db / kWave];
}

// Non-cached tokens x of the lane's request on decodes db .. db+NX-1, as
// fp32, -inf where infeasible.  From the leader row (min with the cap), or
// for a request marked to match on its own, a first-miss scan of its run in
// integers (x then rounded to fp32, as the scoring kernel does).
template <int NX>
__device__ inline void sweep_x(const Snap &s, const Table &t, const Reqs &rq, const Hot &rec, uint32_t r,
                               const float *lead_lam, uint32_t db, float (&xf)[NX]) {
    if ((int32_t)rec.lams >= 0) {
        const float lenf = __uint_as_float(rec.len);
        const float *row = lead_lam + rec.lrow / sizeof(float);
#pragma unroll
        for (int u = 0; u < NX; ++u) {
            const uint32_t d = db + u;
            float x = -__builtin_inff();
            if (d < s.D) {
                const uint64_t xlim = s.dxlim[d];
                const float xm = xlim == 0 ? -1.0f : (float)(xlim - 1 < kExactTok ? xlim - 1 : (uint64_t)kExactTok);
                const float lam = __uint_as_float(min(__float_as_uint(row[d]), rec.lams));
                const float xx = lenf - lam;
                x = xx <= xm ? xx : -__builtin_inff();
            }
            xf[u] = x;
        }
        return;
    }
    uint32_t p, len, n;
    uint64_t a;
    request_ok(rq, s, r, p, len, a, n);   // validated by the selection
    uint32_t jx[NX];
#pragma unroll
    for (int u = 0; u < NX; ++u) jx[u] = n;
    uint64_t alive = ~0ull;
    for (uint32_t b = 0; b < n && alive; ++b) {
        const uint64_t dead = alive & ~held_mask(t, holder_lane(t, rq.hashes[a + b]), db);
#pragma unroll
        for (int u = 0; u < NX; ++u) jx[u] = (dead >> u) & 1ull ? b : jx[u];
        alive &= ~dead;
    }
#pragma unroll
    for (int u = 0; u < NX; ++u) {
        const uint32_t d = db + u;
        float x = -__builtin_inff();
        if (d < s.D) {
            const uint32_t xi = len - s.block_tokens * jx[u];
            x = (uint64_t)xi < s.dxlim[d] ? (float)xi : -__builtin_inff();
        }
        xf[u] = x;
    }
}

// One thread per request (batch order), kSweepScen scenarios per
// workgroup.  LDS: the (L + load term) constants of every (p, d) and two
// buffers of one scenario's seconds per token, rows of Dp = D | 1 (an odd
// pitch, so lanes of different prefills read different banks).  While a
// scenario is scored from one buffer, each thread holds its share of the
// next scenario's table (loaded before the scoring, at most kSweepHold
// entries) and stores it into the other buffer afterwards, so one barrier
// per scenario suffices and the loads' latency is hidden behind the
// scoring; larger tables are copied before each scenario instead.  NX decodes'
// tokens are held in registers; a pool of more decodes is taken NX at a
// time and its tokens recomputed per scenario.  FULL: exactly NX decodes,
// every decode index a compile-time constant (no bounds test per pair).
// Writes the top-k of every scenario and counts, per scenario, the requests
// whose selected tier / decode differs from the loaded snapshot's selection.
template <int K, int NX, bool LDS, bool FULL>
__global__ __launch_bounds__(kSweepThreads, FULL ? (K == 1 ? 6 : 5) : 1) void sweep_kernel(Snap s, Table t, Reqs rq, const Hot *__restrict__ hotr,
                                                             const float *__restrict__ lead_lam,
                                                             const float *__restrict__ spt_scen, uint32_t n_scen,
                                                             const int32_t *__restrict__ base_idx,
                                                             const float *__restrict__ base_score, uint32_t k_out,
                                                             int32_t *__restrict__ out_idx,
                                                             float *__restrict__ out_score,
                                                             unsigned long long *__restrict__ flips) {
    extern __shared__ float tab[];   // LDS: [P][Dp] constants, then 2 x [P][Dp] seconds per token
    const uint32_t P = s.P, D = FULL ? (uint32_t)NX : s.D, Dp = D | 1u;
    const uint32_t r = blockIdx.x * kSweepThreads + threadIdx.x;
    const uint32_t s0 = blockIdx.y * kSweepScen;
    const uint32_t s1 = min(s0 + kSweepScen, n_scen);
    const bool act = r < rq.n_req;
    const bool valid = act && !__builtin_isnan(base_score[r]);
    Hot rec = Hot{0, 0, 0, 0};
    uint32_t p = 0;
    if (valid) {
        rec = hotr[r];
        p = rec.row / (s.slp * (uint32_t)sizeof(float2));
    }
    float *tc = tab, *tsb = tab + (uint64_t)P * Dp;
    // a scenario's seconds per token into LDS buffer b (all of them, by
    // this workgroup's threads)
    auto table_copy = [&](uint32_t sc, uint32_t b) {
        const float *sp = spt_scen + (uint64_t)sc * P * D;
        float *ts = tsb + (uint64_t)b * P * Dp;
        for (uint32_t i = threadIdx.x; i < P * D; i += kSweepThreads) {
            const uint32_t pp = i / D;
            ts[pp * Dp + (i - pp * D)] = sp[i];
        }
    };
    const bool held = P * D <= kSweepThreads * kSweepHold;
    if (LDS) {
        for (uint32_t i = threadIdx.x; i < P * D; i += kSweepThreads) {
            const uint32_t pp = i / D, d = i - pp * D;
            tc[pp * Dp + d] = s.sl[(uint64_t)pp * s.slp + d].y;
        }
        if (held && s0 < s1) table_copy(s0, 0);
    }
    const bool one = FULL || D <= (uint32_t)NX;
    float xf[NX];
    if (valid && one) sweep_x<NX>(s, t, rq, rec, r, lead_lam, 0, xf);
    const int32_t bsel = valid ? base_idx[r] : -1;
    const int btier = bsel < 0 ? -1 : (int)(s.tier_map[(uint64_t)p * D + (uint32_t)bsel] & 3u);
    const uint32_t lrow = p * Dp;
    for (uint32_t sc = s0; sc < s1; ++sc) {
        const float *sp = spt_scen + (uint64_t)sc * P * D;
        const uint32_t buf = held ? (sc - s0) & 1u : 0u;
        const float *ts = tsb + (uint64_t)buf * P * Dp;
        float nx[kSweepHold];   // this thread's share of the next scenario's table
        if (LDS) {
            if (held) {
                __syncthreads();   // this scenario's buffer is written and the other one no longer read
                if (sc + 1 < s1) {
                    const float *spn = sp + (uint64_t)P * D;
#pragma unroll
                    for (uint32_t h = 0; h < kSweepHold; ++h) {
                        const uint32_t i = threadIdx.x + h * kSweepThreads;
                        nx[h] = i < P * D ? spn[i] : 0.0f;
                    }
                }
            } else {
                __syncthreads();   // the previous scenario's table is no longer read
                table_copy(sc, 0);
                __syncthreads();
            }
        }
        uint32_t tk[K], ti[K];
#pragma unroll
        for (int q = 0; q < K; ++q) {
            tk[q] = 0xFFFFFFFFu;
            ti[q] = 0xFFFFFFFFu;
        }
        if (valid) {
            if (FULL) {
#pragma unroll
                for (int u = 0; u < NX; ++u) {
                    const float spt = LDS ? ts[lrow + u] : sp[(uint64_t)p * D + u];
                    const float cst = LDS ? tc[lrow + u] : s.sl[(uint64_t)p * s.slp + u].y;
                    topk_ins32<K>(tk, ti, __float_as_uint(fmaf(xf[u], spt, cst)), (uint32_t)u);
                }
            } else {
                for (uint32_t db = 0; db < D; db += NX) {
                    if (!one) sweep_x<NX>(s, t, rq, rec, r, lead_lam, db, xf);
#pragma unroll
                    for (int u = 0; u < NX; ++u) {
                        const uint32_t d = db + u;
                        if (d < D) {
                            const float spt = LDS ? ts[lrow + d] : sp[(uint64_t)p * D + d];
                            const float cst = LDS ? tc[lrow + d] : s.sl[(uint64_t)p * s.slp + d].y;
                            topk_ins32<K>(tk, ti, __float_as_uint(fmaf(xf[u], spt, cst)), d);
                        }
                    }
                }
            }
        }
        if (LDS && held && sc + 1 < s1) {
            float *tn = tsb + (uint64_t)(buf ^ 1u) * P * Dp;
#pragma unroll
            for (uint32_t h = 0; h < kSweepHold; ++h) {
                const uint32_t i = threadIdx.x + h * kSweepThreads;
                if (i < P * D) {
                    const uint32_t pp = i / D;
                    tn[pp * Dp + (i - pp * D)] = nx[h];
                }
            }
        }
        uint32_t tier_flip = 0, idx_flip = 0;
        if (act) {
            const uint64_t o = ((uint64_t)sc * rq.n_req + r) * k_out;
#pragma unroll
            for (int q = 0; q < K; ++q) {
                if ((uint32_t)q < k_out) {
                    // a key with its sign bit set is an infeasible pair (cost -inf)
                    const bool none = !valid || tk[q] >= 0x80000000u;
                    out_idx[o + q] = none ? -1 : (int32_t)ti[q];
                    out_score[o + q] = !valid ? __builtin_nanf("") : none ? __builtin_inff() : __uint_as_float(tk[q]);
                }
            }
            if (valid) {
                const int32_t sel = tk[0] >= 0x80000000u ? -1 : (int32_t)ti[0];
                const int ts_ = sel < 0 ? -1 : (int)(s.tier_map[(uint64_t)p * D + (uint32_t)sel] & 3u);
                tier_flip = ts_ != btier;
                idx_flip = sel != bsel;
            }
        }
        if (flips) {
            const uint32_t fa = wave_sum_u32(tier_flip), fb = wave_sum_u32(idx_flip);
            if ((threadIdx.x % kWave) == 0) {
                if (fa) atomicAdd(flips + 2 * sc, (unsigned long long)fa);
                if (fb) atomicAdd(flips + 2 * sc + 1, (unsigned long long)fb);
            }
        }
    }
}

// Proposition 2 (Sec. V-D) per scenario: pairs of decodes on different
// tiers from one prefill instance, their bandwidths X = B'(1 - c) with
// B' = B_tau / (1 + n_inflight[tau][p]) under the snapshot's congestion and
// under the scenario's, counted into out[3 s + 0..2]: pairs the
// proposition's sufficient condition covers (the larger of the two
// congestion errors below |X - X'| / (B'_tau + B'_tau')), inverted pairs
// among them, all inverted pairs (the snapshot's strict order not kept).
// fp64, every operation in a fixed order, so the counts are exact.  One
// thread per (p, d), pairs with the decodes after d.
struct Bw64 {
    double b[4];
};

__global__ __launch_bounds__(256) void tier_inv_kernel(Snap s, Bw64 bw, const float *__restrict__ util_scen,
                                                       unsigned long long *__restrict__ out) {
    const uint32_t sc = blockIdx.y;
    const uint64_t pd = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t npd = (uint64_t)s.P * s.D;
    uint32_t covered = 0, inv_cov = 0, inverted = 0;
    if (pd < npd) {
        const uint32_t p = (uint32_t)(pd / s.D), d = (uint32_t)(pd - (uint64_t)p * s.D);
        const float *u = util_scen + (uint64_t)sc * npd;
        // B' of each tier for this prefill (the same division for every pair)
        double bt[4];
#pragma unroll
        for (uint32_t t = 0; t < 4; ++t) bt[t] = bw.b[t] / (1.0 + (double)s.n_inflight[t * s.P + p]);
        const uint32_t ta = s.tier_map[pd] & 3u;
        const double ba = ta == 0 ? bt[0] : ta == 1 ? bt[1] : ta == 2 ? bt[2] : bt[3];
        const double ca = (double)s.util[pd], ha = (double)u[pd];
        const double xa = ba * (1.0 - ca), ya = ba * (1.0 - ha);
        for (uint32_t e = d + 1; e < s.D; ++e) {
            const uint64_t q = (uint64_t)p * s.D + e;
            const uint32_t tb = s.tier_map[q] & 3u;
            if (tb == ta) continue;
            const double bb = tb == 0 ? bt[0] : tb == 1 ? bt[1] : tb == 2 ? bt[2] : bt[3];
            const double cb = (double)s.util[q], hb = (double)u[q];
            const double xb = bb * (1.0 - cb), yb = bb * (1.0 - hb);
            if (xa == xb) continue;
            const bool inv = xa > xb ? !(ya > yb) : !(ya < yb);
            const double eps = fmax(fabs(ha - ca), fabs(hb - cb));
            const bool cov = eps < fabs(xa - xb) / (ba + bb);
            covered += cov;
            inv_cov += cov && inv;
            inverted += inv;
        }
    }
    covered = wave_sum_u32(covered);
    inv_cov = wave_sum_u32(inv_cov);
    inverted = wave_sum_u32(inverted);
    if ((threadIdx.x % kWave) == 0) {
        if (covered) atomicAdd(out + 3 * (uint64_t)sc, (unsigned long long)covered);
        if (inv_cov) atomicAdd(out + 3 * (uint64_t)sc + 1, (unsigned long long)inv_cov);
        if (inverted) atomicAdd(out + 3 * (uint64_t)sc + 2, (unsigned long long)inverted);
    }
}

// ------------------------------------------------------------------ table build

// Sets *flag when the resident hashes hold the reserved value 0.
__global__ void count_zero_kernel(const uint64_t *__restrict__ h, uint64_t n, uint32_t *__restrict__ flag) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    bool z = false;
    for (; i < n; i += stride) z |= h[i] == 0;
    if (__any(z) && (threadIdx.x % kWave) == 0) atomicOr(flag, 1u);
}

// ---- holder index build (once per cache load)
//
// The (hash, decode) pairs of all resident sets are sorted by hash (rocPRIM
// radix sort), so the holders of one hash form a run.  The first element of
// each run ("head") stands for the run: classify_kernel counts distinct
// hashes and those with two or more holders, index_insert_kernel puts every
// distinct hash into the cuckoo set, and index_value_kernel finds each one's
// slot and writes its holder value (for several holders, a fresh bitmap row
// with their bits set).

// Decode of every resident hash of the CSR (binary search of the offsets).
__global__ void owner_kernel(const uint64_t *__restrict__ off, uint32_t D, uint64_t first, uint64_t n,
                             uint32_t *__restrict__ owner) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) {
        const uint64_t x = first + i;
        uint32_t lo = 0, hi = D;   // largest d with off[d] <= x
        while (hi - lo > 1) {
            const uint32_t mid = lo + (hi - lo) / 2;
            if (off[mid] <= x) lo = mid;
            else hi = mid;
        }
        owner[i] = lo;
    }
}

__device__ inline bool run_head(const uint64_t *__restrict__ key, uint64_t i) {
    return i == 0 || key[i] != key[i - 1];
}

// Smallest and largest holder of the run starting at head i; returns the
// run's end.
__device__ inline uint64_t run_span(const uint64_t *__restrict__ key, const uint32_t *__restrict__ dec, uint64_t n,
                                    uint64_t i, uint32_t &dmin, uint32_t &dmax) {
    dmin = dmax = dec[i];
    uint64_t e = i + 1;
    for (; e < n && key[e] == key[i]; ++e) {
        dmin = min(dmin, dec[e]);
        dmax = max(dmax, dec[e]);
    }
    return e;
}

// cnt[0] += distinct hashes, cnt[1] += hashes with two or more holders.
__global__ __launch_bounds__(256) void classify_kernel(const uint64_t *__restrict__ key,
                                                       const uint32_t *__restrict__ dec, uint64_t n,
                                                       unsigned long long *__restrict__ cnt) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    uint32_t heads = 0, multi = 0;
    for (; i < n; i += stride) {
        if (!run_head(key, i)) continue;
        uint32_t dmin, dmax;
        run_span(key, dec, n, i, dmin, dmax);
        ++heads;
        multi += dmin != dmax ? 1u : 0u;
    }
    heads = wave_sum_u32(heads);
    multi = wave_sum_u32(multi);
    if ((threadIdx.x % kWave) == 0) {
        if (heads) atomicAdd(cnt, (unsigned long long)heads);
        if (multi) atomicAdd(cnt + 1, (unsigned long long)multi);
    }
}

// Cuckoo insertion of the distinct hashes.  A key goes to an empty slot of
// either candidate bucket (compare-and-swap 0 -> key); when all four slots
// are taken it displaces the key of a random slot by atomic exchange (a
// random walk: a fresh key picks either bucket, a displaced key its other
// bucket) and carries the displaced key on.  A key is always either in the
// set or carried by exactly one thread, so none is lost.
constexpr uint32_t kMaxKicks = 2048;

__device__ inline bool try_place(unsigned long long *bk, uint64_t key) {
    for (int slot = 0; slot < 2; ++slot) {
        const unsigned long long prev = atomicCAS(bk + slot, 0ull, (unsigned long long)key);
        if (prev == 0ull || prev == key) return true;
    }
    return false;
}

__global__ __launch_bounds__(256) void index_insert_kernel(uint64_t *__restrict__ keys, uint32_t shift,
                                                           const uint64_t *__restrict__ skey, uint64_t n,
                                                           uint32_t *__restrict__ err) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    unsigned long long *tab = (unsigned long long *)keys;
    for (; i < n; i += stride) {
        if (!run_head(skey, i)) continue;
        uint64_t key = skey[i];
        uint32_t from = 0xFFFFFFFFu;   // bucket the carried key was displaced from
        uint32_t rnd = (uint32_t)(key ^ (key >> 32)) ^ (uint32_t)i;   // walk state (a 32-bit LCG)
        bool done = false;
        for (uint32_t kick = 0; kick < kMaxKicks && !done; ++kick) {
            uint32_t b1, b2;
            buckets_of(key, shift, b1, b2);
            if (try_place(tab + 2 * (uint64_t)b1, key) || try_place(tab + 2 * (uint64_t)b2, key)) {
                done = true;
                break;
            }
            // displace from the bucket the key did not just leave; the walk's
            // choices come from the full-period 32-bit LCG of Knuth and Lewis
            // (multiplier 1664525, increment 1013904223; Press et al.,
            // Numerical Recipes, "quick and dirty" generator)
            rnd = rnd * 1664525u + 1013904223u;
            const uint32_t b = (b1 == from) ? b2 : (b2 == from) ? b1 : ((rnd >> 31) ? b2 : b1);
            const unsigned long long old = atomicExch(tab + 2 * (uint64_t)b + ((rnd >> 30) & 1u),
                                                      (unsigned long long)key);
            if (old == 0ull || old == key) {
                done = true;
                break;
            }
            key = old;
            from = b;
        }
        if (!done) atomicOr(err, kErrTableFull);
    }
}

// Holder values, once every key has its final slot.  Bitmap rows are
// handed out by rows_used (row 0 stays zero: the scan reads it when a value
// is not a row); each row is written by the one thread of its run.
__global__ __launch_bounds__(256) void index_value_kernel(const uint64_t *__restrict__ keys, uint32_t *__restrict__ vals,
                                                          uint32_t shift, uint64_t *__restrict__ bits,
                                                          uint32_t bpitch, const uint64_t *__restrict__ skey,
                                                          const uint32_t *__restrict__ dec, uint64_t n,
                                                          uint32_t *__restrict__ rows_used,
                                                          uint32_t *__restrict__ err) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) {
        if (!run_head(skey, i)) continue;
        const uint64_t key = skey[i];
        uint32_t dmin, dmax;
        const uint64_t e = run_span(skey, dec, n, i, dmin, dmax);
        uint32_t v;
        if (dmin == dmax) {
            v = kHeldOne | dmin;
        } else {
            v = atomicAdd(rows_used, 1u);
            uint64_t *row = bits + (uint64_t)v * bpitch;
            for (uint64_t x = i; x < e; ++x) row[dec[x] / 64u] |= 1ull << (dec[x] % 64u);
        }
        uint32_t b1, b2;
        buckets_of(key, shift, b1, b2);
        uint64_t slot = ~0ull;
        if (keys[2 * (uint64_t)b1] == key) slot = 2 * (uint64_t)b1;
        else if (keys[2 * (uint64_t)b1 + 1] == key) slot = 2 * (uint64_t)b1 + 1;
        else if (keys[2 * (uint64_t)b2] == key) slot = 2 * (uint64_t)b2;
        else if (keys[2 * (uint64_t)b2 + 1] == key) slot = 2 * (uint64_t)b2 + 1;
        if (slot == ~0ull) atomicOr(err, kErrTableFull);
        else vals[slot] = v;
    }
}

__global__ void fill_u64_kernel(uint64_t *__restrict__ p, uint64_t n, uint64_t v) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

__global__ void fill_u32_kernel(uint32_t *__restrict__ p, uint64_t n, uint32_t v) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

// ------------------------------------------------------------------ snapshot checks

// Predictive congestion (Sec. VIII): one step of simple exponential
// smoothing of the congestion matrix towards an observation,
// c <- c + beta (obs - c), in fp32.  Both lie in [0, 1) and the result is
// their convex combination, rounded between them, so it stays in [0, 1).
// An observation outside [0, 1) or NaN leaves its entry unchanged and
// raises kErrObservation.
__device__ inline float smooth_one(float u, float o, float beta, bool &bad) {
    if (!(o >= 0.0f && o < 1.0f)) {
        bad = true;
        return u;
    }
    return fmaf(beta, o - u, u);
}

// VEC4: both arrays 16-byte aligned; four entries per thread and step,
// the n % 4 tail by the first threads.
template <bool VEC4>
__global__ __launch_bounds__(256) void smooth_kernel(float *__restrict__ util, const float *__restrict__ obs,
                                                     uint64_t n, float beta, uint32_t *__restrict__ err) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    bool bad = false;
    if (VEC4) {
        const uint64_t n4 = n / 4;
        for (uint64_t v = i; v < n4; v += stride) {
            const float4 o = ((const float4 *)obs)[v];
            float4 u = ((const float4 *)util)[v];
            u.x = smooth_one(u.x, o.x, beta, bad);
            u.y = smooth_one(u.y, o.y, beta, bad);
            u.z = smooth_one(u.z, o.z, beta, bad);
            u.w = smooth_one(u.w, o.w, beta, bad);
            ((float4 *)util)[v] = u;
        }
        i += n4 * 4;
        if (i >= n4 * 4 + 4) i = n;   // only the first threads take the tail
    }
    for (; i < n; i += stride) util[i] = smooth_one(util[i], obs[i], beta, bad);
    if (__ballot(bad) && (threadIdx.x % kWave) == 0) atomicOr(err, kErrObservation);
}

__global__ void check_snapshot_kernel(const uint8_t *__restrict__ tier, const float *__restrict__ util,
                                      uint64_t npd, const uint32_t *__restrict__ batch, uint32_t D,
                                      uint32_t beta_max, uint32_t *__restrict__ bad) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    uint32_t f = 0;
    for (uint64_t x = i; x < npd; x += stride) {
        if (tier && tier[x] > 3) f |= 1u;
        float u = util[x];
        if (!(u >= 0.0f && u < 1.0f)) f |= 2u;
    }
    if (batch)
        for (uint64_t x = i; x < D; x += stride)
            if (batch[x] > beta_max) f |= 4u;
    if (f) atomicOr(bad, f);
}

// ------------------------------------------------------------------ between-batch update

// First-miss scan of one (hash run, decode) pair by one thread.
__device__ inline uint32_t prefix_match_one(const Table &t, uint32_t d, const uint64_t *__restrict__ run,
                                            uint32_t n) {
    uint32_t j = 0;
    while (j < n && holds(t, run[j], d)) ++j;
    return j;
}

__global__ void commit_count_kernel(Snap s, Table t, Reqs rq, const int32_t *__restrict__ sel,
                                    uint32_t *__restrict__ cnt, uint32_t *__restrict__ adm,
                                    unsigned long long *__restrict__ bytes, uint32_t *__restrict__ err) {
    uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rq.n_req) return;
    int32_t d = sel[r];
    if (d < 0) return;
    if ((uint32_t)d >= s.D) {
        atomicOr(err, kErrSelection);
        return;
    }
    uint32_t p, len, n;
    uint64_t a;
    if (!request_ok(rq, s, r, p, len, a, n)) {
        atomicOr(err, kErrRequest);
        return;
    }
    uint32_t j = prefix_match_one(t, (uint32_t)d, rq.hashes + a, n);
    uint64_t s_eff = (uint64_t)s.bpt * (uint64_t)(len - s.block_tokens * j);
    uint32_t tau = s.tier_map[(uint64_t)p * s.D + (uint32_t)d] & 3u;
    atomicAdd(cnt + tau * s.P + p, 1u);
    atomicAdd(adm + d, 1u);
    atomicAdd(bytes + d, (unsigned long long)s_eff);
}

__global__ void commit_apply_kernel(uint32_t P, uint32_t D, uint32_t cap, uint32_t mu,
                                    const uint32_t *__restrict__ cnt, const uint32_t *__restrict__ adm,
                                    const unsigned long long *__restrict__ bytes,
                                    uint16_t *__restrict__ n_inflight, uint32_t *__restrict__ queue,
                                    uint64_t *__restrict__ free_mem, uint64_t *__restrict__ adm_prev) {
    uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 4 * P) n_inflight[i] = (uint16_t)(cnt[i] < cap ? cnt[i] : cap);
    if (i < D) {
        int64_t nq = (int64_t)queue[i] + (int64_t)adm[i] - (int64_t)mu;
        queue[i] = (uint32_t)(nq < 0 ? 0 : nq);
        uint64_t m = free_mem[i], b = bytes[i];
        m = m > b ? m - b : 0;
        free_mem[i] = m + adm_prev[i];
        adm_prev[i] = b;
    }
}

// ---------------------------------------------------------------- tier counts

// Two-hop routing: the route each selection takes (1: staged, 0: direct,
// -1: no selection or an invalid request): the selected pair's prefix
// length (first miss of the run on that decode), then its direct and
// staged costs from the derived rows, in the scoring kernel's arithmetic.
__global__ __launch_bounds__(256) void route_of_kernel(Snap s, Table t, Reqs rq, uint32_t k,
                                                       const int32_t *__restrict__ idx, int8_t *__restrict__ out) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (uint64_t)rq.n_req * k) return;
    const uint32_t r = (uint32_t)(i / k);
    const int32_t d = idx[i];
    uint32_t p, len, n;
    uint64_t a;
    if (d < 0 || (uint32_t)d >= s.D || !request_ok(rq, s, r, p, len, a, n)) {
        out[i] = -1;
        return;
    }
    uint32_t j = 0;
    while (j < n && holds(t, rq.hashes[a + j], (uint32_t)d)) ++j;
    const float x = (float)(len - s.block_tokens * j);
    const uint64_t o = (uint64_t)p * s.slp + (uint32_t)d;
    const float2 r1 = s.sl[o], r2 = s.sr[o];
    out[i] = fmaf(x, r2.x, r2.y) < fmaf(x, r1.x, r1.y) ? 1 : 0;
}

// Non-cached bytes of each selection (Eq. (2) in the integer form
// bpt * (l_r - B_tok * j)): the selected pair's prefix length by the first
// miss of the run on that decode.  0 for no selection or an invalid
// request; a selection index >= D is flagged.
__global__ __launch_bounds__(256) void selection_bytes_kernel(Snap s, Table t, Reqs rq, uint32_t k,
                                                              const int32_t *__restrict__ idx,
                                                              uint64_t *__restrict__ out, uint32_t *__restrict__ err) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (uint64_t)rq.n_req * k) return;
    const uint32_t r = (uint32_t)(i / k);
    const int32_t d = idx[i];
    uint32_t p, len, n;
    uint64_t a;
    if (d >= 0 && (uint32_t)d >= s.D) atomicOr(err, kErrSelection);
    if (d < 0 || (uint32_t)d >= s.D || !request_ok(rq, s, r, p, len, a, n)) {
        out[i] = 0;
        return;
    }
    uint32_t j = 0;
    while (j < n && holds(t, rq.hashes[a + j], (uint32_t)d)) ++j;
    out[i] = (uint64_t)s.bpt * (uint64_t)(len - s.block_tokens * j);
}

// Requests per tier of the selected decode (index 4: rejected), the tier
// shift statistic.  Invalid selections are flagged and not counted.
__global__ __launch_bounds__(256) void tier_count_kernel(Snap s, Reqs rq, const int32_t *__restrict__ sel,
                                                         unsigned long long *__restrict__ counts,
                                                         uint32_t *__restrict__ err) {
    __shared__ uint32_t local[5];
    if (threadIdx.x < 5) local[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < rq.n_req) {
        const int32_t d = sel[r];
        const uint32_t p = rq.prefill[r];
        if (d < 0) {
            atomicAdd(&local[4], 1u);
        } else if ((uint32_t)d < s.D && p < s.P) {
            atomicAdd(&local[s.tier_map[(uint64_t)p * s.D + (uint32_t)d] & 3u], 1u);
        } else {
            atomicOr(err, kErrSelection);
        }
    }
    __syncthreads();
    if (threadIdx.x < 5 && local[threadIdx.x]) atomicAdd(counts + threadIdx.x, (unsigned long long)local[threadIdx.x]);
}

// ---------------------------------------------------------------- sequential selection
//
// Algorithm 1 applied request after request in batch order: the in-flight
// counter of the chosen tier grows by one (up to the cap) before the next
// request from the same prefill instance is scored.  Requests of different
// prefill instances do not interact, so each prefill instance's requests are
// a sequential chain run by one workgroup.  The prefix lengths come from the
// batch selection's scoring records (by batch index) and leader rows: the
// chain reads min(leader row, B_tok * L*) per decode, as the scoring kernel
// does, and no per-pair buffer is written.

// start/end of each prefill instance's run in the order sorted by prefill
__global__ void segment_kernel(const uint32_t *__restrict__ keys, uint32_t n, uint32_t P, uint32_t *__restrict__ start,
                               uint32_t *__restrict__ end) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t k = keys[i];
    if (k >= P) return;
    if (i == 0 || keys[i - 1] != k) start[k] = i;
    if (i + 1 == n || keys[i + 1] != k) end[k] = i + 1;
}

__global__ void prefill_key_kernel(Reqs rq, uint32_t P, const uint32_t *__restrict__ order_keys,
                                   uint32_t *__restrict__ keys, uint32_t *__restrict__ vals) {
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rq.n_req) return;
    keys[r] = order_keys[r] == kKeyInvalid ? P : rq.prefill[r];
    vals[r] = r;
}

// Non-cached tokens x (Eq. (2)) of request r on decodes d0 + stride * k,
// k < M, from its scoring record: the leader row capped by B_tok * L*, or,
// for a request marked to match on its own, a first-miss scan of its hash
// run over the holder index.  Integers throughout (a record's fp32 values
// are integers below 2^24, so exact).  Decodes at or past D get len; the
// caller never finds them feasible.
template <int M>
__device__ inline void seq_tokens(const Snap &s, const Table &t, const Reqs &rq, const Hot *__restrict__ hotr,
                                  const float *__restrict__ lead_lam, uint32_t r, uint32_t d0, uint32_t stride,
                                  uint32_t (&x)[M]) {
    const Hot rec = hotr[r];
    if ((int32_t)rec.lams >= 0) {
        const uint32_t len = (uint32_t)__uint_as_float(rec.len);
        const float *row = lead_lam + rec.lrow / sizeof(float);
#pragma unroll
        for (int k = 0; k < M; ++k) {
            const uint32_t d = d0 + stride * k;
            const uint32_t lam = d < s.D ? min(__float_as_uint(row[d]), rec.lams) : 0u;
            x[k] = len - (uint32_t)__uint_as_float(lam);
        }
        return;
    }
    uint32_t p, len, n;
    uint64_t a;
    request_ok(rq, s, r, p, len, a, n);   // validated by the selection
    uint32_t j[M];
    uint32_t alive = 0;
#pragma unroll
    for (int k = 0; k < M; ++k) {
        j[k] = n;
        alive |= (d0 + stride * k < s.D ? 1u : 0u) << k;
    }
    for (uint32_t b = 0; b < n && alive; ++b) {
        const uint32_t v = holder_lane(t, rq.hashes[a + b]);
#pragma unroll
        for (int k = 0; k < M; ++k) {
            const uint32_t d = d0 + stride * k;
            if (((alive >> k) & 1u) && !((held_mask(t, v, d & ~(uint32_t)(kWave - 1)) >> (d % kWave)) & 1ull)) {
                j[k] = b;
                alive &= ~(1u << k);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < M; ++k) x[k] = len - s.block_tokens * j[k];
}

constexpr int kSeqThreads = 256;

constexpr int kSeqChunk = 8;   // decodes per thread per pass of the general chain

__global__ __launch_bounds__(kSeqThreads) void sequential_kernel(Snap s, Table t, Reqs rq, uint32_t cap,
                                                                 const Hot *__restrict__ hotr,
                                                                 const float *__restrict__ lead_lam,
                                                                 const uint32_t *__restrict__ order,
                                                                 const uint32_t *__restrict__ start,
                                                                 const uint32_t *__restrict__ end,
                                                                 int32_t *__restrict__ out_idx,
                                                                 float *__restrict__ out_score) {
    __shared__ float n_tier[4];
    __shared__ uint32_t best_cost[kSeqThreads / kWave];
    __shared__ uint32_t best_d[kSeqThreads / kWave];
    const uint32_t p = blockIdx.x;
    const uint32_t i0 = start[p], i1 = end[p];
    if (i0 >= i1) return;
    const uint32_t lane = threadIdx.x % kWave, wave = wave_index();
    if (threadIdx.x < 4) n_tier[threadIdx.x] = (float)s.n_inflight[threadIdx.x * s.P + p];
    __syncthreads();
    for (uint32_t i = i0; i < i1; ++i) {
        const uint32_t r = order[i];
        uint32_t lb = 0xFFFFFFFFu, ld = 0xFFFFFFFFu;
        for (uint32_t d0 = threadIdx.x; d0 < s.D; d0 += kSeqThreads * kSeqChunk) {
            uint32_t xc[kSeqChunk];
            seq_tokens<kSeqChunk>(s, t, rq, hotr, lead_lam, r, d0, kSeqThreads, xc);
#pragma unroll
            for (int k = 0; k < kSeqChunk; ++k) {
                const uint32_t d = d0 + kSeqThreads * k, x = xc[k];
                if (d < s.D && (uint64_t)x < s.dxlim[d]) {
                    const uint64_t o = (uint64_t)p * s.D + d;
                    const uint32_t tau = s.tier_map[o] & 3u;
                    const float cost = pair_score(x, sec_per_token_n(s, tau, n_tier[tau], s.util[o]), s.lat[tau],
                                                  s.dbase[d]);
                    const uint32_t cbits = __float_as_uint(cost);
                    if (cbits < lb) {   // d grows within a thread: first strict minimum wins ties
                        lb = cbits;
                        ld = d;
                    }
                }
            }
        }
        const uint32_t mn = wave_min_u32_dpp(lb);
        const uint32_t dm = wave_min_u32_dpp(lb == mn ? ld : 0xFFFFFFFFu);
        if (lane == 0) {
            best_cost[wave] = mn;
            best_d[wave] = dm;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t bc = best_cost[0], bd = best_d[0];
            for (int w = 1; w < kSeqThreads / kWave; ++w)
                if (best_cost[w] < bc || (best_cost[w] == bc && best_d[w] < bd)) {
                    bc = best_cost[w];
                    bd = best_d[w];
                }
            if (bc == 0xFFFFFFFFu) {
                out_idx[r] = -1;
                out_score[r] = __builtin_inff();
            } else {
                out_idx[r] = (int32_t)bd;
                out_score[r] = __uint_as_float(bc);
                const uint32_t tau = s.tier_map[(uint64_t)p * s.D + bd] & 3u;
                if (n_tier[tau] < (float)cap) n_tier[tau] += 1.0f;
            }
        }
        __syncthreads();
    }
}

// One of four uniform values by a per-lane index, without indexing an array.
__device__ inline float pick4(const float (&v)[4], uint32_t t) {
    const float lo = (t & 1u) ? v[1] : v[0];
    const float hi = (t & 1u) ? v[3] : v[2];
    return (t & 2u) ? hi : lo;
}

// The same chain with each thread's decodes (d = thread + T*k, k < MAXC)
// held in registers: tier (2 bits each in one word), seconds per token,
// tier latency plus load term, and the feasibility limit (32 bits, with a
// bit for limits of 2^32 and more, which every x meets); the prefill row's
// congestion sits in LDS.  Between requests only the factors of the tier
// whose counter grew change, and they are recomputed with the same
// expression.
//
// Pipeline: the chain's scoring records (and batch indices) are staged in
// LDS T at a time, two chunks deep, so a request's record is an LDS read;
// the leader-row values of the next request are loaded while the current
// one is scored (raw bits, into the other of two buffers).  Each wave's
// minimum carries the winner's decode and tier (d << 2 | tier), the waves'
// minima go to alternating LDS slots and every thread picks the winner, so
// one barrier per request suffices (a wave can write a slot again only
// after the barrier that follows every wave's reading of it) and the
// counter update needs no memory read.
template <int MAXC>
struct SeqBuf {
    uint32_t raw[MAXC];   // leader-row bits B_tok * j, or B_tok * j itself (own scan)
    uint32_t len, lams, own, r;
};

template <int T, int MAXC>
__global__ __launch_bounds__(T) void sequential_cached_kernel(Snap s, Table t, Reqs rq, uint32_t cap,
                                                              const Hot *__restrict__ hotr,
                                                              const float *__restrict__ lead_lam,
                                                              const uint32_t *__restrict__ order,
                                                              const uint32_t *__restrict__ start,
                                                              const uint32_t *__restrict__ end,
                                                              int32_t *__restrict__ out_idx,
                                                              float *__restrict__ out_score) {
    static_assert(MAXC <= 16, "two tier bits per decode in one word");
    constexpr int NW = T / kWave;
    __shared__ uint32_t slot_c[2][NW], slot_d[2][NW];
    __shared__ Hot crec[2][T];
    __shared__ uint32_t cr[2][T];
    // per thread-decode (index k * T + thread), each entry only ever used by
    // its own thread: the congestion, and a staging area for seconds per
    // token (set-up, counter updates) or an own scan's B_tok * j
    __shared__ float urow[T * MAXC];
    __shared__ uint32_t stage[T * MAXC];
    const uint32_t p = blockIdx.x;
    const uint32_t i0 = start[p], i1 = end[p];
    if (i0 >= i1) return;
    const uint32_t lane = threadIdx.x % kWave, wave = wave_index();
    const uint64_t row = (uint64_t)p * s.D;
    float n_tier[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) n_tier[q] = (float)s.n_inflight[q * s.P + p];
    uint32_t tmask = 0;
    float sk[MAXC], lk[MAXC], xm[MAXC];
    // the factors, one decode at a time through LDS (keeps the divisions'
    // temporaries out of the register budget)
#pragma unroll 1
    for (int k = 0; k < MAXC; ++k) {
        const uint32_t d = threadIdx.x + T * k;
        const uint32_t dd = d < s.D ? d : 0;
        const uint32_t tq = s.tier_map[row + dd] & 3u;
        const float u = s.util[row + dd];
        urow[k * T + threadIdx.x] = u;
        stage[k * T + threadIdx.x] = __float_as_uint(sec_per_token_n(s, tq, pick4(n_tier, tq), u));
        tmask |= tq << (2 * k);
    }
#pragma unroll
    for (int k = 0; k < MAXC; ++k) {
        const uint32_t d = threadIdx.x + T * k;
        const bool ok = d < s.D;
        const uint32_t dd = ok ? d : 0;
        sk[k] = __uint_as_float(stage[k * T + threadIdx.x]);
        lk[k] = tier_latency(s, (tmask >> (2 * k)) & 3u) + s.dbase[dd];
        // the largest feasible token count, as fp32 (exact: capped at 2^24,
        // beyond every count of the fp32 path); -1 when nothing is feasible
        // (and for decodes past D, never chosen)
        const uint64_t xl = ok ? s.dxlim[dd] : 0;
        xm[k] = xl == 0 ? -1.0f : (float)(xl - 1 < kExactTok ? xl - 1 : (uint64_t)kExactTok);
    }
    // stage chunk c (positions i0 + c*T ...) of the chain's records in LDS
    auto fill = [&](uint32_t c) {
        const uint32_t i = i0 + c * T + threadIdx.x;
        if (i < i1) {
            const uint32_t r = order[i];
            crec[c & 1u][threadIdx.x] = hotr[r];
            cr[c & 1u][threadIdx.x] = r;
        }
    };
    // read position i's record and start loading its leader-row values
    auto issue = [&](uint32_t i, SeqBuf<MAXC> &b) {
        const uint32_t o = i - i0, c = o / T;
        if (o % T == 0 && c >= 1) fill(c + 1);   // chunk c-1's last record was read before the last barrier
        const Hot &h = crec[c & 1u][o % T];
        const uint32_t r = __builtin_amdgcn_readfirstlane(cr[c & 1u][o % T]);
        const uint32_t lams = __builtin_amdgcn_readfirstlane(h.lams);
        b.r = r;
        if ((int32_t)lams >= 0) {
            const float *lrow = lead_lam + __builtin_amdgcn_readfirstlane(h.lrow) / sizeof(float);
            b.len = (uint32_t)__uint_as_float(__builtin_amdgcn_readfirstlane(h.len));
            b.lams = lams;
            b.own = 0;
#pragma unroll
            for (int k = 0; k < MAXC; ++k) {
                // decodes past D read decode 0's value; their limit 0 makes them infeasible
                const uint32_t d = threadIdx.x + T * k;
                b.raw[k] = __float_as_uint(lrow[d < s.D ? d : 0u]);
            }
        } else {
            // matched on its own: a first-miss scan of its run per decode, in
            // integers, B_tok * j through LDS
            uint32_t pp, len, n;
            uint64_t a;
            request_ok(rq, s, r, pp, len, a, n);   // validated by the selection
#pragma unroll 1
            for (int k = 0; k < MAXC; ++k) {
                const uint32_t d = threadIdx.x + T * k;
                uint32_t j = n;
                if (d < s.D) {
                    const uint32_t db = d & ~(uint32_t)(kWave - 1), bit = d % kWave;
                    for (uint32_t bk = 0; bk < n; ++bk)
                        if (!((held_mask(t, holder_lane(t, rq.hashes[a + bk]), db) >> bit) & 1ull)) {
                            j = bk;
                            break;
                        }
                }
                stage[k * T + threadIdx.x] = s.block_tokens * j;
            }
            b.len = len;
            b.lams = 0xFFFFFFFFu;
            b.own = 1;
#pragma unroll
            for (int k = 0; k < MAXC; ++k) b.raw[k] = stage[k * T + threadIdx.x];
        }
    };
    // score the buffered request, choose, count the choice
    auto step = [&](uint32_t i, const SeqBuf<MAXC> &b) {
        // the lane's least cost bits and the k of its decode: from the leader
        // row in fp32 (token counts below 2^24 are exact, as in the scoring
        // kernel), or for a request matched on its own in integers
        uint32_t lb = 0xFFFFFFFFu, kf = 0;
        if (!b.own) {
            const float lenf = (float)b.len;
#pragma unroll
            for (int k = 0; k < MAXC; ++k) {
                const float x = lenf - __uint_as_float(min(b.raw[k], b.lams));
                const uint32_t c = __float_as_uint(fmaf(x, sk[k], lk[k]));
                if (x <= xm[k] && c < lb) {   // d grows with k: the first strict minimum wins ties
                    lb = c;
                    kf = (uint32_t)k;
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < MAXC; ++k) {
                const uint32_t d = threadIdx.x + T * k;
                const uint32_t x = b.len - b.raw[k];
                if (d < s.D && (uint64_t)x < s.dxlim[d < s.D ? d : 0]) {
                    const uint32_t c = __float_as_uint(fmaf((float)x, sk[k], lk[k]));
                    if (c < lb) {
                        lb = c;
                        kf = (uint32_t)k;
                    }
                }
            }
        }
        const uint32_t ld = lb == 0xFFFFFFFFu ? 0xFFFFFFFFu
                                              : ((threadIdx.x + T * kf) << 2) | ((tmask >> (2 * kf)) & 3u);
        const uint32_t mn = wave_min_u32_dpp(lb);
        const uint32_t dm = wave_min_u32_dpp(lb == mn ? ld : 0xFFFFFFFFu);
        const uint32_t sl = i & 1u;
        if (lane == 0) {
            slot_c[sl][wave] = mn;
            slot_d[sl][wave] = dm;
        }
        __syncthreads();
        uint32_t bc = slot_c[sl][0], bd = slot_d[sl][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            const uint32_t c = slot_c[sl][w], dw = slot_d[sl][w];
            if (c < bc || (c == bc && dw < bd)) {
                bc = c;
                bd = dw;
            }
        }
        if (threadIdx.x == 0) {
            out_idx[b.r] = bc == 0xFFFFFFFFu ? -1 : (int32_t)(bd >> 2);
            out_score[b.r] = bc == 0xFFFFFFFFu ? __builtin_inff() : __uint_as_float(bc);
        }
        if (bc != 0xFFFFFFFFu) {
            const uint32_t tw = bd & 3u;
            const float nw = pick4(n_tier, tw);
            if (nw < (float)cap) {
                // at most cap times per tier: the tier's factors again, with
                // the same expression, through LDS
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if ((uint32_t)q == tw) n_tier[q] = nw + 1.0f;
#pragma unroll
                for (int k = 0; k < MAXC; ++k) stage[k * T + threadIdx.x] = __float_as_uint(sk[k]);
#pragma unroll 1
                for (int k = 0; k < MAXC; ++k)
                    if (((tmask >> (2 * k)) & 3u) == tw)
                        stage[k * T + threadIdx.x] =
                            __float_as_uint(sec_per_token_n(s, tw, nw + 1.0f, urow[k * T + threadIdx.x]));
#pragma unroll
                for (int k = 0; k < MAXC; ++k) sk[k] = __uint_as_float(stage[k * T + threadIdx.x]);
            }
        }
    };
    fill(0);
    fill(1);
    __syncthreads();
    SeqBuf<MAXC> ba, bb;
    issue(i0, ba);
    for (uint32_t i = i0; i < i1; i += 2) {
        if (i + 1 < i1) issue(i + 1, bb);
        step(i, ba);
        if (i + 1 >= i1) break;
        if (i + 2 < i1) issue(i + 2, ba);
        step(i + 1, bb);
    }
}

// Work buffers of one selection: per-request ordering buffers and records,
// the leader table, the leaders' holder values, per-group partial top-k
// keys and the sort / scan temporaries.  Owned by the handle (grown on
// demand, or sized ahead by netkv_reserve) or carved from the library's
// static scratch array (netkv_select_batch_noalloc).
struct Scratch {
    uint64_t order_cap = 0;   // requests the per-request buffers hold
    uint32_t *keys_in = nullptr, *keys_out = nullptr, *vals_in = nullptr, *perm = nullptr;
    Hot *hot = nullptr;       // [order_cap + kHotPad] scoring-order records, the part every step reads
    Cold *cold = nullptr;     // and the request's index in the batch
    uint64_t *seg = nullptr;    // in-tile inclusive scan of the positions' (leader, L) elements, hash order
    uint64_t *tpre = nullptr;   // per order tile: its total, then the exclusive prefix of the tiles before it
    Pre *hrec = nullptr;      // prefill row and length by hash-order position
    Cold *crec = nullptr;
    uint32_t *pkey = nullptr, *pkey_out = nullptr, *pval = nullptr, *pord = nullptr;   // prefill order
    uint32_t *n_valid = nullptr;
    unsigned long long *hv_used = nullptr;
    unsigned int *n_lead = nullptr;
    uint32_t *hv = nullptr;   // holder values of the leaders' blocks
    uint64_t hv_cap = 0;
    Lead *lead = nullptr;     // leader table
    float *lead_lam = nullptr;   // [lead_cap + 1][D] B_tok * prefix length of each leader;
                                 // row lead_cap is all zero (no leader)
    uint32_t lead_cap = 0, lead_D = 0;
    bool zero_row_set = false;   // row lead_cap has been cleared
    void *sort_tmp = nullptr;    // rocPRIM sort / scan temporary storage
    size_t sort_tmp_bytes = 0;
    // the batch sorts' own buffers: digit counts, totals and the ping-pong
    // pair (null when the per-request buffers hold no more than kSortMinN)
    uint32_t *sort_cnt = nullptr, *sort_tot = nullptr, *keys_tmp = nullptr, *vals_tmp = nullptr;
    uint64_t *partial = nullptr;   // [groups][R][K] per-group top-k keys
    uint64_t partial_cap = 0;
    Hot *hotr = nullptr;           // scoring records by batch index (ranking sweep, sequential form)
    uint64_t hotr_cap = 0;
};

}  // namespace

// ====================================================================== host side

constexpr uint32_t kTimeSlots = 256;   // timed launches kept for netkv_kernel_ms

struct netkv_ctx {
    int device = 0;
    std::string err;
    // snapshot
    bool have_snap = false;
    uint32_t P = 0, D = 0;
    uint8_t *tier_map = nullptr;
    float *util = nullptr;
    uint16_t *n_inflight = nullptr;
    uint64_t *free_mem = nullptr;
    uint32_t *queue = nullptr;
    uint32_t *batch = nullptr;
    uint64_t *adm_prev = nullptr;
    float2 *sl = nullptr;        // derived per call: [P*D]
    float *dbase = nullptr;      // [D]
    uint64_t *dxlim = nullptr;   // [D]
    float bw[4] = {0, 0, 0, 0}, lat[4] = {0, 0, 0, 0};
    double bw64[4] = {0, 0, 0, 0};   // the snapshot's bandwidths as given (Proposition 2's counts)
    // a second stream (default priority, non-blocking) on which a large
    // selection runs the derivation and the leader kernels beside the
    // ordering kernels, forked from and joined to the caller's stream by
    // events (so a caller's graph capture takes both branches)
    hipStream_t side = nullptr;
    hipEvent_t ev_fork0 = nullptr, ev_fork1 = nullptr, ev_join = nullptr;
    // the ranking sweep's fork of Proposition 2's counts onto the same stream
    hipEvent_t ev_inv_fork = nullptr, ev_inv_join = nullptr;
    // the flow simulation's work buffer (flowsim.hip)
    void *flow_buf = nullptr;
    uint64_t flow_buf_bytes = 0;
    float t_a = 0, t_b = 0, alpha = 0;
    uint32_t beta_max = 0, bpt = 0, block_tokens = 1;
    uint64_t m_min = 0;
    // cache
    bool have_cache = false;
    uint32_t cache_D = 0;
    // holder index of the resident sets
    uint64_t *table = nullptr;   // [buckets][2] distinct resident hashes
    uint32_t *tvals = nullptr;   // [buckets][2] holder values
    uint64_t *bits = nullptr;    // [rows][bpitch] holder bitmaps
    uint64_t table_bytes = 0, buckets = 0, rows = 0, distinct = 0;
    uint32_t log2b = 0, bpitch = 0;
    // scratch
    uint32_t *errword = nullptr;          // request / selection errors (sticky)
    uint32_t *loadword = nullptr;         // validation flags of the load calls
    float *spt_scen = nullptr;    // ranking sweep: seconds per token of every (scenario, p, d)
    uint64_t spt_cap = 0;
    int32_t *base_idx = nullptr;
    float *base_score = nullptr;
    uint64_t base_n = 0;
    uint32_t *cnt = nullptr, *adm = nullptr;
    unsigned long long *bytes = nullptr;
    uint32_t commit_P = 0, commit_D = 0;
    // work buffers of the selection (grow to the largest batch seen)
    Scratch sc;
    // options
    uint32_t run_len_opt = 0;   // 0 = automatic
    uint32_t reuse_opt = 1;     // share prefix lengths along the hash order
    uint32_t lead_cap_opt = 0;  // leader table limit (0 = by memory)
    uint32_t cols_opt = 0;      // decodes per lane (0 = automatic)
    uint32_t policy_opt = 0;    // 0 full, 1 without live congestion, 2 topology only
    // sequential-selection scratch
    uint32_t *seq_keys = nullptr, *seq_vals = nullptr, *seq_keys_out = nullptr, *seq_perm = nullptr;
    uint32_t *seq_start = nullptr, *seq_end = nullptr;
    uint64_t seq_cap = 0;
    uint32_t seq_P = 0;
    // timing
    bool timing = false;
    // two-hop routing: the staged route's hop tiers and congestion per (p, d),
    // and its derived rows (like sl)
    uint8_t *rt1 = nullptr, *rt2 = nullptr;
    float *ru1 = nullptr, *ru2 = nullptr;
    float2 *sr = nullptr;
    bool have_route = false;
    // kernel timing: begin/end event pairs in a ring, created on first enable
    std::vector<hipEvent_t> tev;
    uint32_t tcount = 0;    // launches timed since timing was enabled
};

namespace {

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

// Events around the one timed kernel of an API call (when timing is on).
hipError_t time_begin(netkv_handle h, hipStream_t st) {
    if (!h->timing) return hipSuccess;
    return hipEventRecord(h->tev[2 * (h->tcount % kTimeSlots)], st);
}

hipError_t time_end(netkv_handle h, hipStream_t st) {
    if (!h->timing) return hipSuccess;
    const hipError_t e = hipEventRecord(h->tev[2 * (h->tcount % kTimeSlots) + 1], st);
    if (e == hipSuccess) ++h->tcount;
    return e;
}

// Timing suspended for a scope (inner steps of a call that times another kernel).
struct TimingOff {
    netkv_handle h;
    bool was;
    explicit TimingOff(netkv_handle hh) : h(hh), was(hh->timing) { h->timing = false; }
    ~TimingOff() { h->timing = was; }
};

netkv_status fail(netkv_handle h, netkv_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (h) h->err = buf;
    return st;
}

#define HIPCHK(h, call)                                                                        \
    do {                                                                                       \
        hipError_t e_ = (call);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail((h), e_ == hipErrorOutOfMemory ? NETKV_ENOMEM : NETKV_EDEVICE,         \
                        "%s failed: %s", #call, hipGetErrorString(e_));                        \
    } while (0)

template <typename T>
void dfree(T *&p) {
    if (p) (void)hipFree((void *)p);
    p = nullptr;
}

template <typename T>
hipError_t dalloc(T *&p, uint64_t count) {
    dfree(p);
    void *q = nullptr;
    hipError_t e = hipMalloc(&q, std::max<uint64_t>(count, 1) * sizeof(T));
    p = (T *)q;
    return e;
}

uint32_t grid_for(uint64_t n, uint32_t block, uint32_t maxg = 1u << 16) {
    uint64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > maxg) g = maxg;
    return (uint32_t)g;
}

Snap make_snap(netkv_handle h) {
    Snap s;
    s.tier_map = h->tier_map;
    s.util = h->util;
    s.n_inflight = h->n_inflight;
    s.free_mem = h->free_mem;
    s.queue = h->queue;
    s.batch = h->batch;
    for (int i = 0; i < 4; ++i) {
        s.bw[i] = h->bw[i];
        s.lat[i] = h->lat[i];
    }
    s.t_a = h->t_a;
    s.t_b = h->t_b;
    s.alpha = h->alpha;
    s.beta_max = h->beta_max;
    s.m_min = h->m_min;
    s.bpt = h->bpt;
    s.block_tokens = h->block_tokens;
    s.P = h->P;
    s.D = h->D;
    s.sl = h->sl;
    s.slp = sl_pitch(h->D);
    s.sr = nullptr;
    s.dbase = h->dbase;
    s.dxlim = h->dxlim;
    s.policy = h->policy_opt;
    return s;
}

Table make_table(netkv_handle h) {
    Table t;
    t.keys = h->table;
    t.vals = h->tvals;
    t.bits = h->bits;
    t.shift = 64 - h->log2b;
    t.bpitch = h->bpitch;
    return t;
}

netkv_status check_requests(netkv_handle h, const netkv_requests_t *req) {
    if (!req) return fail(h, NETKV_EINVAL, "requests is NULL");
    if (req->n_req && (!req->prefill || !req->len_tokens || !req->hash_off))
        return fail(h, NETKV_EINVAL, "request arrays must not be NULL");
    if (req->n_req && req->n_hashes && !req->hashes) return fail(h, NETKV_EINVAL, "hashes is NULL");
    if (req->n_req > (1u << 31)) return fail(h, NETKV_EINVAL, "n_req too large");
    return NETKV_OK;
}

Reqs make_reqs(const netkv_requests_t *req) {
    Reqs r;
    r.n_req = req->n_req;
    r.prefill = req->prefill;
    r.len = req->len_tokens;
    r.off = req->hash_off;
    r.hashes = req->hashes;
    r.n_hashes = req->n_hashes;
    return r;
}

netkv_status ready(netkv_handle h) {
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded (netkv_oracle_load)");
    if (!h->have_cache) return fail(h, NETKV_ENOTREADY, "no cache loaded (netkv_cache_load)");
    if (h->cache_D != h->D)
        return fail(h, NETKV_EINVAL, "cache has %u decodes, snapshot %u", h->cache_D, h->D);
    return NETKV_OK;
}

// rocPRIM's radix sorts of the batch-order keys (batches outside the range
// of the own batch sort): its tuned kernels, with the merge-sort path
// limited to 2^16 items (rocPRIM's own limit is 2^20).  Above the limit
// the onesweep radix sort takes one pass per 8 key bits; measured on
// MI355X at 2^20 requests, 91 us for the 11-bit prefill order against
// 150 us for the block sort and twenty merge passes.
using SortConfig = rocprim::radix_sort_config<rocprim::default_config, rocprim::default_config,
                                              rocprim::default_config, (size_t)1 << 16>;

// Leader table capacity: prefix lengths of at most 256 MiB (u32 per decode),
// and no more leaders than requests.  Leaders beyond it (and the requests
// that follow them) are matched on their own by the scoring kernel.
constexpr uint64_t kLeadBytes = 256ull << 20;

uint32_t lead_capacity(uint64_t R, uint32_t D) {
    const uint64_t c = std::min<uint64_t>(std::max<uint64_t>(R, 1), kLeadBytes / (4ull * D));
    return (uint32_t)std::max<uint64_t>(c, 1);
}

uint32_t bits_for(uint64_t v) {   // bits to hold 0..v
    uint32_t b = 1;
    while (b < 64 && (v >> b)) ++b;
    return b;
}

void free_scratch(Scratch &sc) {
    dfree(sc.keys_in); dfree(sc.keys_out); dfree(sc.vals_in); dfree(sc.perm); dfree(sc.hot); dfree(sc.cold);
    dfree(sc.seg); dfree(sc.tpre); dfree(sc.hrec); dfree(sc.crec);
    dfree(sc.pkey); dfree(sc.pkey_out); dfree(sc.pval); dfree(sc.pord);
    dfree(sc.n_valid); dfree(sc.hv_used); dfree(sc.n_lead); dfree(sc.hv); dfree(sc.lead); dfree(sc.lead_lam);
    dfree(sc.sort_tmp); dfree(sc.sort_cnt); dfree(sc.sort_tot); dfree(sc.keys_tmp); dfree(sc.vals_tmp);
    dfree(sc.partial);
    dfree(sc.hotr);
    sc = Scratch();
}

// rocPRIM temporary storage for the batch orders of R requests (both sorts
// share one buffer); a size query only.
hipError_t sort_tmp_bytes_for(uint64_t R, size_t &bytes) {
    size_t b1 = 0, b2 = 0;
    uint32_t *k = nullptr;
    hipError_t err = rocprim::radix_sort_pairs<SortConfig>(nullptr, b1, k, k, k, k, (uint32_t)R, 0, 32, nullptr);
    if (err == hipSuccess)
        err = rocprim::radix_sort_pairs<SortConfig>(nullptr, b2, k, k, k, k, (uint32_t)R, 0, 32, nullptr);
    bytes = std::max<size_t>(std::max(b1, b2), 16);
    return err;
}

// The handle's work buffers for a batch of R requests with n_hashes block
// hashes and partial_elems per-group keys: grown (never shrunk) when a batch
// needs more than any earlier one or than netkv_reserve provided.
netkv_status ensure_scratch(netkv_handle h, Scratch &sc, uint64_t R, uint64_t partial_elems, uint64_t n_hashes,
                            hipStream_t st) {
    if (R > sc.order_cap) {
        dfree(sc.keys_in); dfree(sc.keys_out); dfree(sc.vals_in); dfree(sc.perm); dfree(sc.hot); dfree(sc.cold);
        dfree(sc.seg); dfree(sc.tpre); dfree(sc.pkey); dfree(sc.pkey_out); dfree(sc.pval); dfree(sc.pord);
        dfree(sc.hrec); dfree(sc.crec);
        dfree(sc.sort_tmp);
        dfree(sc.sort_cnt); dfree(sc.sort_tot); dfree(sc.keys_tmp); dfree(sc.vals_tmp);
        sc.order_cap = 0;
        sc.sort_tmp_bytes = 0;
        if (dalloc(sc.keys_in, R) != hipSuccess || dalloc(sc.keys_out, R) != hipSuccess ||
            dalloc(sc.vals_in, R) != hipSuccess || dalloc(sc.perm, R) != hipSuccess ||
            dalloc(sc.hot, R + kHotPad) != hipSuccess || dalloc(sc.cold, R) != hipSuccess ||
            dalloc(sc.seg, R) != hipSuccess || dalloc(sc.tpre, R / kOrderPos + 1) != hipSuccess ||
            dalloc(sc.pkey, R) != hipSuccess || dalloc(sc.pkey_out, R) != hipSuccess ||
            dalloc(sc.pval, R) != hipSuccess || dalloc(sc.pord, R) != hipSuccess ||
            dalloc(sc.hrec, R) != hipSuccess || dalloc(sc.crec, R) != hipSuccess)
            return fail(h, NETKV_ENOMEM, "batch scratch allocation failed");
        // one temporary buffer for the two sorts and the scan
        size_t bytes = 0;
        if (sort_tmp_bytes_for(R, bytes) != hipSuccess) return fail(h, NETKV_EDEVICE, "sort / scan size query failed");
        uint8_t *tmp = nullptr;
        if (dalloc(tmp, bytes) != hipSuccess) return fail(h, NETKV_ENOMEM, "sort scratch allocation failed");
        sc.sort_tmp = tmp;
        sc.sort_tmp_bytes = bytes;
        if (R > kSortMinN) {
            // the own batch sorts run for kSortMinN < n <= kSortMaxN
            const uint64_t n = std::min<uint64_t>(R, kSortMaxN);
            // the most tiles of any batch up to n: small tiles up to
            // kSortSmallTileN, large beyond
            const uint64_t ns = std::min<uint64_t>(n, kSortSmallTileN);
            const uint64_t ntile = std::max((ns + kSortSmallTile - 1) / kSortSmallTile, (n + kSortTile - 1) / kSortTile);
            if (dalloc(sc.sort_cnt, ntile * kSortMaxBins) != hipSuccess ||
                dalloc(sc.sort_tot, kSortMaxBins) != hipSuccess || dalloc(sc.keys_tmp, n) != hipSuccess ||
                dalloc(sc.vals_tmp, n) != hipSuccess)
                return fail(h, NETKV_ENOMEM, "sort scratch allocation failed");
        }
        sc.order_cap = R;
    }
    if (!sc.n_valid && dalloc(sc.n_valid, 1) != hipSuccess) return fail(h, NETKV_ENOMEM, "allocation failed");
    if (!sc.hv_used && dalloc(sc.hv_used, 1) != hipSuccess) return fail(h, NETKV_ENOMEM, "allocation failed");
    if (!sc.n_lead && dalloc(sc.n_lead, 1) != hipSuccess) return fail(h, NETKV_ENOMEM, "allocation failed");
    // holder values of the leaders' blocks: at most one per block of the
    // batch (fewer if runs overlap in the hash array; leaders that do not
    // fit look their blocks up in the leader kernel)
    if (n_hashes > sc.hv_cap || !sc.hv) {
        dfree(sc.hv);
        sc.hv_cap = 0;
        if (dalloc(sc.hv, std::max<uint64_t>(n_hashes, 1)) != hipSuccess)
            return fail(h, NETKV_ENOMEM, "holder value scratch allocation failed");
        sc.hv_cap = std::max<uint64_t>(n_hashes, 1);
    }
    const uint32_t lc = lead_capacity(R, h->D);
    if (lc > sc.lead_cap || sc.lead_D != h->D || !sc.lead) {
        dfree(sc.lead);
        dfree(sc.lead_lam);
        sc.lead_cap = 0;
        sc.zero_row_set = false;
        if (dalloc(sc.lead, lc) != hipSuccess || dalloc(sc.lead_lam, (uint64_t)(lc + 1) * h->D + kRowPad) != hipSuccess)
            return fail(h, NETKV_ENOMEM, "leader table allocation failed");
        sc.lead_cap = lc;
        sc.lead_D = h->D;
    }
    if (partial_elems > sc.partial_cap) {
        dfree(sc.partial);
        sc.partial_cap = 0;
        if (dalloc(sc.partial, partial_elems) != hipSuccess)
            return fail(h, NETKV_ENOMEM, "partial top-k scratch allocation failed");
        sc.partial_cap = partial_elems;
    }
    return NETKV_OK;
}

// One pass of the batch sort over key bits [shift, shift + bits): counts,
// offsets, scatter (ASSEMBLE: the prefill order's scoring records).
template <bool ASSEMBLE>
hipError_t sort_pass(netkv_handle h, Scratch &sc, const uint32_t *kin, const uint32_t *vin, uint32_t *kout,
                     uint32_t *vout, uint32_t n, uint32_t shift, uint32_t bits, const Pre *hrec,
                     const uint64_t *seg, const uint64_t *tpre, const Cold *crec, uint32_t lstride, uint32_t zrow,
                     Hot *hot, Cold *cold, Hot *hotr, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const uint32_t tile = sort_tile(n);
    const uint32_t ntile = (n + tile - 1) / tile;   // <= kColPer * kBlock (n <= kSortMaxN)
    if (tile == kSortSmallTile)
        hipLaunchKernelGGL(sort_count_kernel<kSortSmallTile>, dim3(ntile), dim3(kBlock), 0, st, kin, n, shift, bits,
                           sc.sort_cnt);
    else
        hipLaunchKernelGGL(sort_count_kernel<kSortTile>, dim3(ntile), dim3(kBlock), 0, st, kin, n, shift, bits,
                           sc.sort_cnt);
    hipLaunchKernelGGL(sort_colscan_kernel, dim3(1u << bits), dim3(kBlock), 0, st, sc.sort_cnt, ntile, bits,
                       sc.sort_tot);
    if (tile == kSortSmallTile)
        hipLaunchKernelGGL((sort_scatter_kernel<ASSEMBLE, kSortSmallTile>), dim3(ntile), dim3(kBlock), 0, st, kin,
                           vin, n, shift, bits, (const uint32_t *)sc.sort_cnt, (const uint32_t *)sc.sort_tot, kout,
                           vout, hrec, seg, tpre, crec, h->block_tokens, lstride, zrow, hot, cold, hotr);
    else
        hipLaunchKernelGGL((sort_scatter_kernel<ASSEMBLE, kSortTile>), dim3(ntile), dim3(kBlock), 0, st, kin, vin,
                           n, shift, bits, (const uint32_t *)sc.sort_cnt, (const uint32_t *)sc.sort_tot, kout, vout,
                           hrec, seg, tpre, crec, h->block_tokens, lstride, zrow, hot, cold, hotr);
    return hipGetLastError();
}

// Bits of pass p of `passes` even passes over nbits key bits, and its shift.
inline void pass_bits(uint32_t nbits, uint32_t passes, uint32_t p, uint32_t &shift, uint32_t &bits) {
    shift = 0;
    for (uint32_t q = 0; q <= p; ++q) {
        bits = (nbits - shift + (passes - q) - 1) / (passes - q);
        if (q < p) shift += bits;
    }
    bits = std::max(bits, 1u);
}

// Stable sort of n (key, value) pairs on key bits [0, nbits) (values: vin,
// or the input positions when vin is null), in passes of at most
// kSortPassBits through the handle's ping-pong buffers; the result lands in
// kout / vout (kSortMinN < n <= kSortMaxN).
hipError_t batch_sort_pairs(netkv_handle h, Scratch &sc, const uint32_t *kin, const uint32_t *vin, uint32_t *kout,
                            uint32_t *vout, uint32_t n, uint32_t nbits, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const uint32_t passes = std::max(1u, (nbits + kSortPassBits - 1) / kSortPassBits);
    const uint32_t *sk = kin, *sv = vin;
    for (uint32_t p = 0; p < passes; ++p) {
        uint32_t shift, bits;
        pass_bits(nbits, passes, p, shift, bits);
        // the last pass writes kout, the one before the ping-pong buffers, ...
        const bool to_out = ((passes - 1 - p) % 2) == 0;
        uint32_t *dk = to_out ? kout : sc.keys_tmp, *dv = to_out ? vout : sc.vals_tmp;
        const hipError_t e = sort_pass<false>(h, sc, sk, sv, dk, dv, n, shift, bits, nullptr, nullptr, nullptr,
                                              nullptr, 0, 0, nullptr, nullptr, nullptr, st);
        if (e != hipSuccess) return e;
        sk = dk;
        sv = dv;
    }
    return hipSuccess;
}

// The prefill order: a stable sort of the hash-order positions by the
// prefill key (pbits <= kPrefillMaxBits), whose last pass writes the
// scoring records at their output positions; earlier passes go through
// buf_k / buf_v (free at this point of a selection).
hipError_t prefill_order(netkv_handle h, Scratch &sc, uint32_t n, uint32_t pbits, uint32_t *buf_k,
                         uint32_t *buf_v, uint32_t lstride, uint32_t zrow, Hot *hotr, hipStream_t st) {
    const uint32_t passes = std::max(1u, (pbits + kSortMaxBits - 1) / kSortMaxBits);
    const uint32_t *sk = sc.pkey, *sv = nullptr;
    for (uint32_t p = 0; p < passes; ++p) {
        uint32_t shift, bits;
        pass_bits(pbits, passes, p, shift, bits);
        hipError_t e;
        if (p + 1 == passes) {
            e = sort_pass<true>(h, sc, sk, sv, nullptr, nullptr, n, shift, bits, sc.hrec, sc.seg, sc.tpre, sc.crec,
                                lstride, zrow, sc.hot, sc.cold, hotr, st);
        } else {
            uint32_t *dk = (p % 2) ? buf_k : sc.keys_tmp, *dv = (p % 2) ? buf_v : sc.vals_tmp;
            e = sort_pass<false>(h, sc, sk, sv, dk, dv, n, shift, bits, nullptr, nullptr, nullptr, nullptr, 0, 0,
                                 nullptr, nullptr, nullptr, st);
            sk = dk;
            sv = dv;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

uint32_t auto_run_len(uint64_t R, uint32_t ngroup) {
    // runs of 128 sorted requests, shortened (to 8 at least) while that
    // leaves fewer than 32K wavefronts (measured on MI355X: 1,048,576
    // requests of 25 blocks on 8 decode groups score fastest in runs of
    // 128, 65,536 wavefronts, against 64, which starts more runs with a
    // full scan, and 256; 262,144 requests of 191 blocks fastest in runs of
    // 64, 32,768 wavefronts, against 32 and 128)
    const uint64_t work = R * ngroup;
    uint64_t rl = 128;
    while (rl > 8 && work / rl < 32768) rl /= 2;
    return (uint32_t)rl;
}

// decodes per lane (or the option: 1, 2, 3, 4 or 6): the widest of 6, 3
// and 2 whose groups of 64 * C decodes split evenly over the XCDs (at least
// one each), so that every XCD's L2 keeps its own slice of the snapshot
// rows; else 2 on pools of 256+ decodes, else 1 (measured on MI355X: wider
// groups share each request's scalar work over more decodes; 12 per lane
// spills registers, and merging the groups of 3,072 decodes in one
// workgroup was slower than XCD-sliced groups and a merge kernel)
inline uint32_t cols_per_lane(uint32_t D, uint32_t opt) {
    if (opt == 1 || opt == 2 || opt == 3 || opt == 4 || opt == 6) return opt;
    for (uint32_t c : {6u, 3u, 2u}) {
        const uint32_t g = (D + kWave * c - 1) / (kWave * c);
        if (g >= kXcds && g % kXcds == 0) return c;
    }
    return D >= 4u * kWave ? 2u : 1u;
}

// The scoring kernel.  A pool of one group of one
// decode per lane (up to 64 decodes) is scored in merged mode: one
// wavefront per run, writing its requests' outputs itself.  Otherwise one
// workgroup per
// (kWavesPerBlock runs, group) when the groups split evenly over the XCDs
// (see score_kernel), else per kWavesPerBlock waves, writing per-group keys
// that reduce_kernel merges.
template <int K, int C>
hipError_t launch_score(netkv_handle h, Scratch &sc, const Snap &sn, const Table &t, const Reqs &rq,
                        const Order &ord, uint32_t run_len, uint32_t n_runs, uint32_t ngroup, const PairOut &po,
                        bool pairs, uint32_t k, int32_t *idx, float *score, hipStream_t st) {
    hipError_t e = time_begin(h, st);
    if (e != hipSuccess) return e;
    constexpr bool kMergeable = C == 1;
    const bool merge = kMergeable && ngroup == 1;
    const uint64_t grid64 = merge ? (uint64_t)(n_runs + kXcds - 1) / kXcds * kXcds
                            : ngroup % kXcds == 0
                                ? (uint64_t)((n_runs + kWavesPerBlock - 1) / kWavesPerBlock) * ngroup
                                : ((uint64_t)n_runs * ngroup + kWavesPerBlock - 1) / kWavesPerBlock;
    const uint32_t grid = (uint32_t)grid64;
    const uint32_t block = merge ? ngroup * kWave : kBlock;
    // a request that matches on its own (its leader did not fit the leader
    // table, or 2^24 tokens or more) looks blocks up one at a time: rare,
    // and a short loop keeps the kernel's registers for the common path
    const bool two = sn.sr != nullptr;
#define NETKV_SCORE(P2, T2, M2)                                                                                  \
    hipLaunchKernelGGL((score_kernel<K, 1, C, P2, T2, M2>), dim3(grid), dim3(block), 0, st, sn, t, ord.hot,     \
                       ord.cold, ord.lam, sc.lead_cap + 1, rq.hashes, rq.len, rq.off, ord.n_valid, rq.n_req,      \
                       run_len, n_runs, ngroup, sc.partial, po, k, idx, score)
    if (merge) {
        if (pairs) {
            if (two) NETKV_SCORE(true, true, kMergeable);
            else NETKV_SCORE(true, false, kMergeable);
        } else {
            if (two) NETKV_SCORE(false, true, kMergeable);
            else NETKV_SCORE(false, false, kMergeable);
        }
    } else {
        if (pairs) {
            if (two) NETKV_SCORE(true, true, false);
            else NETKV_SCORE(true, false, false);
        } else {
            if (two) NETKV_SCORE(false, true, false);
            else NETKV_SCORE(false, false, false);
        }
    }
#undef NETKV_SCORE
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = time_end(h, st)) != hipSuccess || merge) return e;
    hipLaunchKernelGGL((reduce_kernel<K>), dim3((rq.n_req + 255) / 256), dim3(256), 0, st, rq.n_req, ngroup, k,
                       (const uint64_t *)sc.partial, (const Cold *)ord.cold, ord.n_valid, idx, score);
    return hipGetLastError();
}

// The scoring kernel (bracketed by the handle's timing events when
// enabled), then, outside merged mode, the merge.
template <int K>
hipError_t launch_score_reduce(netkv_handle h, Scratch &sc, const Snap &sn, const Table &t, const Reqs &rq,
                               const Order &ord, uint32_t run_len, uint32_t n_runs, uint32_t ngroup, uint32_t C,
                               const PairOut &po, bool pairs, uint32_t k, int32_t *idx, float *score,
                               hipStream_t st) {
    switch (C) {
    case 6: return launch_score<K, 6>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, po, pairs, k, idx, score, st);
    case 4: return launch_score<K, 4>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, po, pairs, k, idx, score, st);
    case 3: return launch_score<K, 3>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, po, pairs, k, idx, score, st);
    case 2: return launch_score<K, 2>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, po, pairs, k, idx, score, st);
    default: return launch_score<K, 1>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, po, pairs, k, idx, score, st);
    }
}

// Top-k width K of the kernels for k, decodes per lane C and decode groups.
struct Geometry {
    uint32_t K, C, ngroup;
};

Geometry geometry(netkv_handle h, uint32_t k) {
    Geometry g;
    g.K = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : 8;
    g.C = cols_per_lane(h->D, h->cols_opt);
    g.ngroup = (h->D + kWave * g.C - 1) / (kWave * g.C);
    return g;
}

// The whole selection of one batch on `st` with the work buffers of sc
// (which must hold the batch: R <= order_cap, R * ngroup * K <= partial_cap):
// validate and key the requests, hash order (sort), common runs and
// leaders, the segmented scan, prefill order (stable sort), scoring
// records, leaders' prefix lengths, scoring, merge.  Launches kernels only.
netkv_status run_select(netkv_handle h, Scratch &sc, const netkv_requests_t *req, uint32_t k, int32_t *idx,
                        float *score, const PairOut &po, bool pairs, uint32_t max_blocks, hipStream_t st,
                        bool route2 = false, bool derive = true, Hot *hotr = nullptr) {
    const uint64_t R = req->n_req;
    const Geometry geo = geometry(h, k);
    const uint32_t K = geo.K, C = geo.C, ngroup = geo.ngroup;
    Snap sn = make_snap(h);
    const Table t = make_table(h);
    const Reqs rq = make_reqs(req);
    if (!sc.zero_row_set) {
        // the all-zero row of requests without a leader (no leader writes it)
        hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(h->D, 256)), dim3(256), 0, st,
                           (uint32_t *)(sc.lead_lam + (uint64_t)sc.lead_cap * h->D), (uint64_t)h->D, 0u);
        HIPCHK(h, hipGetLastError());
        sc.zero_row_set = true;
    }
    // a large batch forks a second stream: the derivation (independent of
    // the ordering), then after the order kernel the leaders' holder values
    // and prefix lengths, beside the tile prefixes and the prefill order;
    // joined before the scoring kernel
    const bool fork = R >= kForkMinN;
    hipStream_t s2 = fork ? h->side : st;
    if (fork) {
        HIPCHK(h, hipEventRecord(h->ev_fork0, st));
        HIPCHK(h, hipStreamWaitEvent(s2, h->ev_fork0, 0));
    }
    const uint64_t nd = std::max<uint64_t>((uint64_t)h->P * h->D, h->D);
    if (derive)
        hipLaunchKernelGGL(derive_kernel, dim3((uint32_t)((nd + 255) / 256)), dim3(256), 0, s2, sn, h->sl, h->dbase,
                           h->dxlim);
    if (route2 && h->have_route) {
        if (derive)
            hipLaunchKernelGGL(derive_route_kernel, dim3((uint32_t)((nd + 255) / 256)), dim3(256), 0, s2, sn,
                               (const uint8_t *)h->rt1, (const float *)h->ru1, (const uint8_t *)h->rt2,
                               (const float *)h->ru2, h->sr);
        sn.sr = h->sr;
    }
    // the own batch sort (its first pass takes positions as values) where
    // its buffers are there and the batch is in its range
    const bool own_sort = R > kSortMinN && R <= kSortMaxN && sc.sort_cnt != nullptr;
    hipLaunchKernelGGL(prep_kernel, dim3((uint32_t)((R + 255) / 256)), dim3(256), 0, st, sn, rq, max_blocks,
                       sc.keys_in, own_sort ? nullptr : sc.vals_in, h->errword, sc.hv_used, sc.n_lead, k, idx, score);
    HIPCHK(h, hipGetLastError());
    size_t tb = sc.sort_tmp_bytes;
    if (own_sort)
        HIPCHK(h, batch_sort_pairs(h, sc, sc.keys_in, nullptr, sc.keys_out, sc.perm, (uint32_t)R, 32, st));
    else
        HIPCHK(h, rocprim::radix_sort_pairs<SortConfig>(sc.sort_tmp, tb, sc.keys_in, sc.keys_out, sc.vals_in,
                                                        sc.perm, (uint32_t)R, 0, 32, st));
    // leaders (and holder values of their blocks) the table takes this call
    const uint32_t lcap = h->lead_cap_opt ? std::min(sc.lead_cap, h->lead_cap_opt) : sc.lead_cap;
    const uint64_t hvcap = h->lead_cap_opt ? std::min<uint64_t>(sc.hv_cap, h->lead_cap_opt) : sc.hv_cap;
    // the prefill order: the own sort (positions as its values), or rocPRIM's on pval
    const uint32_t pbits = bits_for(h->P);
    const bool own_prefill = own_sort && pbits <= kPrefillMaxBits;
    hipLaunchKernelGGL(order_kernel<kLcpLanes>, dim3((uint32_t)((R * kLcpLanes + 255) / 256)), dim3(256), 0, st, rq,
                       h->P, sl_pitch(h->D), h->block_tokens, (const uint32_t *)sc.perm,
                       (const uint32_t *)sc.keys_out, t, h->reuse_opt, sc.seg, sc.tpre, sc.pkey,
                       own_prefill ? nullptr : sc.pval, sc.hrec, sc.crec, sc.lead, lcap, sc.n_lead, hvcap,
                       sc.hv_used, sc.n_valid);
    HIPCHK(h, hipGetLastError());
    if (fork) {
        HIPCHK(h, hipEventRecord(h->ev_fork1, st));
        HIPCHK(h, hipStreamWaitEvent(s2, h->ev_fork1, 0));
    }
    hipLaunchKernelGGL(lead_holder_kernel, dim3((uint32_t)std::min<uint64_t>((lcap + kWavesPerBlock - 1) /
                                                                             kWavesPerBlock, 4096)),
                       dim3(kBlock), 0, s2, t, rq.hashes, sc.lead, (const unsigned int *)sc.n_lead, lcap, sc.hv);
    {
        // leaders' prefix lengths: 64 decodes per wavefront, 64 blocks per step
        const uint32_t lgroup = (h->D + kWave - 1) / kWave;
        const uint64_t lw = std::min<uint64_t>((uint64_t)lcap * ((lgroup + kLeadGroups - 1) / kLeadGroups), 65536);
        hipLaunchKernelGGL(lead_kernel, dim3((uint32_t)((lw + kWavesPerBlock - 1) / kWavesPerBlock)),
                           dim3(kBlock), 0, s2, t, h->D, h->block_tokens, (const Lead *)sc.lead,
                           (const unsigned int *)sc.n_lead, lcap, (const uint32_t *)sc.hv, rq.hashes, lgroup,
                           sc.lead_lam);
    }
    HIPCHK(h, hipGetLastError());
    // the exclusive prefixes of the order tiles' totals (the second level of
    // the segmented scan; the first is in order_kernel)
    hipLaunchKernelGGL(tile_prefix_kernel, dim3(1), dim3(kPrefixThreads), 0, st, sc.tpre,
                       (uint32_t)((R + kOrderPos - 1) / kOrderPos));
    HIPCHK(h, hipGetLastError());
    // prefill order (stable: the hash order within each prefill) and the
    // scoring records in it
    const uint32_t lstride = h->D * (uint32_t)sizeof(float);
    if (own_prefill) {
        // (the hash order's keys and permutation are no longer needed)
        HIPCHK(h, prefill_order(h, sc, (uint32_t)R, pbits, sc.keys_out, sc.perm, lstride, sc.lead_cap * lstride,
                                hotr, st));
    } else {
        tb = sc.sort_tmp_bytes;
        HIPCHK(h, rocprim::radix_sort_pairs<SortConfig>(sc.sort_tmp, tb, sc.pkey, sc.pkey_out, sc.pval, sc.pord,
                                                        (uint32_t)R, 0, pbits, st));
        hipLaunchKernelGGL(assemble_kernel, dim3((uint32_t)((R + kHotPad + 255) / 256)), dim3(256), 0, st,
                           (uint32_t)R, h->block_tokens, lstride, sc.lead_cap * lstride, (const uint32_t *)sc.pord,
                           (const uint64_t *)sc.seg, (const uint64_t *)sc.tpre, (const Pre *)sc.hrec,
                           (const Cold *)sc.crec, sc.hot, sc.cold, hotr);
        HIPCHK(h, hipGetLastError());
    }
    if (fork) {
        HIPCHK(h, hipEventRecord(h->ev_join, s2));
        HIPCHK(h, hipStreamWaitEvent(st, h->ev_join, 0));
    }
    const uint32_t run_len = h->run_len_opt ? h->run_len_opt : auto_run_len(R, ngroup);
    const uint32_t n_runs = (uint32_t)((R + run_len - 1) / run_len);
    Order ord{sc.hot, sc.cold, sc.lead_lam, sc.hv, sc.n_valid, lcap};
    if (K == 1)
        HIPCHK(h, launch_score_reduce<1>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, C, po, pairs, k, idx,
                                         score, st));
    else if (K == 2)
        HIPCHK(h, launch_score_reduce<2>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, C, po, pairs, k, idx,
                                         score, st));
    else if (K == 4)
        HIPCHK(h, launch_score_reduce<4>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, C, po, pairs, k, idx,
                                         score, st));
    else
        HIPCHK(h, launch_score_reduce<8>(h, sc, sn, t, rq, ord, run_len, n_runs, ngroup, C, po, pairs, k, idx,
                                         score, st));
    return NETKV_OK;
}

// Scoring records by batch index for n requests (ranking sweep, sequential form).
netkv_status ensure_hotr(netkv_handle h, uint64_t n) {
    if (n <= h->sc.hotr_cap) return NETKV_OK;
    dfree(h->sc.hotr);
    h->sc.hotr_cap = 0;
    if (dalloc(h->sc.hotr, n) != hipSuccess) return fail(h, NETKV_ENOMEM, "record scratch allocation failed");
    h->sc.hotr_cap = n;
    return NETKV_OK;
}

// The sequential form's per-prefill ordering of R requests over P prefill
// instances (seq), and the ranking sweep's selection under the loaded
// snapshot (base).
netkv_status ensure_seq(netkv_handle h, uint64_t R, uint64_t P, bool seq, bool base) {
    if (seq && h->seq_cap < R) {
        dfree(h->seq_keys); dfree(h->seq_vals); dfree(h->seq_keys_out); dfree(h->seq_perm);
        h->seq_cap = 0;
        HIPCHK(h, dalloc(h->seq_keys, R));
        HIPCHK(h, dalloc(h->seq_vals, R));
        HIPCHK(h, dalloc(h->seq_keys_out, R));
        HIPCHK(h, dalloc(h->seq_perm, R));
        h->seq_cap = R;
    }
    if (seq && h->seq_P != P) {
        dfree(h->seq_start); dfree(h->seq_end);
        h->seq_P = 0;
        HIPCHK(h, dalloc(h->seq_start, P));
        HIPCHK(h, dalloc(h->seq_end, P));
        h->seq_P = (uint32_t)P;
    }
    if (base && h->base_n < R) {
        dfree(h->base_idx);
        dfree(h->base_score);
        h->base_n = 0;
        HIPCHK(h, dalloc(h->base_idx, R));
        HIPCHK(h, dalloc(h->base_score, R));
        h->base_n = R;
    }
    return NETKV_OK;
}

// The handle's buffers for the batch, then the selection.
// With want_hotr, every request's scoring record is also kept by batch
// index in sc.hotr (grown to the batch).
netkv_status select_owned(netkv_handle h, const netkv_requests_t *req, uint32_t k, int32_t *idx, float *score,
                          const PairOut &po, bool pairs, uint32_t max_blocks, hipStream_t st, bool route2 = false,
                          bool want_hotr = false) {
    const Geometry geo = geometry(h, k);
    netkv_status e = ensure_scratch(h, h->sc, req->n_req, (uint64_t)req->n_req * geo.ngroup * geo.K,
                                    req->n_hashes, st);
    if (e) return e;
    if (want_hotr && (e = ensure_hotr(h, req->n_req))) return e;
    return run_select(h, h->sc, req, k, idx, score, po, pairs, max_blocks, st, route2, true,
                      want_hotr ? h->sc.hotr : nullptr);
}

// ---- work buffers carved from the static scratch array (no allocation)

constexpr uint64_t kAlign = 256;
inline uint64_t align_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Lay out the buffers of a selection of at most r requests (no own-sort
// buffers: r <= kSortMinN), lead_cap leaders and hv_cap holder values in
// the bytes at base; with base null only the size is computed.  Returns
// the bytes used.
uint64_t carve(uint8_t *base, uint64_t r, uint32_t D, uint64_t partial_elems, uint32_t lead_cap, uint64_t hv_cap,
               size_t tmp_bytes, Scratch *sc) {
    uint64_t used = 0;
    auto take = [&](uint64_t bytes) -> uint8_t * {
        uint8_t *p = base ? base + used : nullptr;
        used = align_up(used + std::max<uint64_t>(bytes, 1));
        return p;
    };
    Scratch t;
    t.n_valid = (uint32_t *)take(4);
    t.hv_used = (unsigned long long *)take(8);
    t.n_lead = (unsigned int *)take(4);
    t.sort_tmp = take(tmp_bytes);
    t.sort_tmp_bytes = tmp_bytes;
    t.keys_in = (uint32_t *)take(4 * r);
    t.keys_out = (uint32_t *)take(4 * r);
    t.vals_in = (uint32_t *)take(4 * r);
    t.perm = (uint32_t *)take(4 * r);
    t.hot = (Hot *)take(sizeof(Hot) * (r + kHotPad));
    t.cold = (Cold *)take(sizeof(Cold) * r);
    t.seg = (uint64_t *)take(8 * r);
    t.tpre = (uint64_t *)take(8 * (r / kOrderPos + 1));
    t.hrec = (Pre *)take(sizeof(Pre) * r);
    t.crec = (Cold *)take(sizeof(Cold) * r);
    t.pkey = (uint32_t *)take(4 * r);
    t.pkey_out = (uint32_t *)take(4 * r);
    t.pval = (uint32_t *)take(4 * r);
    t.pord = (uint32_t *)take(4 * r);
    t.partial = (uint64_t *)take(8 * partial_elems);
    t.partial_cap = partial_elems;
    t.lead = (Lead *)take(sizeof(Lead) * (uint64_t)lead_cap);
    t.lead_lam = (float *)take(4ull * (((uint64_t)lead_cap + 1) * D + kRowPad));
    t.lead_cap = lead_cap;
    t.lead_D = D;
    t.hv = (uint32_t *)take(4 * hv_cap);
    t.hv_cap = hv_cap;
    t.order_cap = r;
    t.zero_row_set = false;
    if (sc) *sc = t;
    return used;
}

// Sub-batch size and buffers for a no-allocation selection of R requests:
// the largest r (at most kSortMinN, halved down to 256) whose per-request
// buffers and per-group keys fit with one leader row; what is left goes
// half to leader rows, half to leaders' holder values.
netkv_status carve_static(netkv_handle h, uint8_t *base, uint64_t R, uint32_t k, Scratch &sc, uint64_t &r_sub) {
    const Geometry geo = geometry(h, k);
    const uint32_t D = h->D;
    uint64_t r = std::min<uint64_t>(R, kSortMinN);
    size_t tmp = 0;
    for (;;) {
        if (sort_tmp_bytes_for(r, tmp) != hipSuccess) return fail(h, NETKV_EDEVICE, "sort / scan size query failed");
        if (carve(nullptr, r, D, r * geo.ngroup * geo.K, 1, 1, tmp, nullptr) <= kScratchBytes) break;
        if (r <= 256)
            return fail(h, NETKV_ECAPACITY,
                        "the no-allocation scratch (%llu MiB) cannot hold a sub-batch of %llu requests on %u decodes "
                        "with k = %u",
                        (unsigned long long)(kScratchBytes >> 20), (unsigned long long)r, D, k);
        r = std::max<uint64_t>(256, r / 2);
    }
    const uint64_t base_bytes = carve(nullptr, r, D, r * geo.ngroup * geo.K, 1, 1, tmp, nullptr);
    const uint64_t rest = kScratchBytes - base_bytes;
    const uint64_t row = 4ull * D + sizeof(Lead);
    const uint64_t slack = 4 * kAlign;
    uint64_t extra = rest > slack ? std::min<uint64_t>(r - 1, (rest - slack) / 2 / row) : 0;
    uint64_t hv_cap = 1 + (rest > slack + extra * row ? (rest - slack - extra * row) / 4 : 0);
    while (carve(nullptr, r, D, r * geo.ngroup * geo.K, (uint32_t)(1 + extra), hv_cap, tmp, nullptr) > kScratchBytes) {
        if (hv_cap > 1024) hv_cap -= 1024;
        else if (extra > 0) --extra;
        else break;   // one leader row and one holder value: fits (checked above)
    }
    carve(base, r, D, r * geo.ngroup * geo.K, (uint32_t)(1 + extra), hv_cap, tmp, &sc);
    r_sub = r;
    return NETKV_OK;
}

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

}  // namespace

namespace {

template <int K, int NX, bool LDS, bool FULL>
void launch_sweep(dim3 grid, size_t lds, hipStream_t st, const Snap &sn, const Table &t, const Reqs &rq,
                  const Hot *hotr, const float *lead_lam, const float *spt, uint32_t n_scen, const int32_t *bidx,
                  const float *bsc, uint32_t k, int32_t *out_idx, float *out_score, unsigned long long *fl) {
    hipLaunchKernelGGL((sweep_kernel<K, NX, LDS, FULL>), grid, dim3(kSweepThreads), lds, st, sn, t, rq, hotr,
                       lead_lam, spt, n_scen, bidx, bsc, k, out_idx, out_score, fl);
}

// 48 decodes (the 64-GPU pools) with compile-time decode indices, up to 48
// with a bounds test, more 64 at a time; the per-(p, d) tables in LDS when
// they fit, else read from memory.
template <int K>
void launch_sweep_k(uint32_t D, bool lds, dim3 grid, size_t lds_bytes, hipStream_t st, const Snap &sn, const Table &t,
                    const Reqs &rq, const Hot *hotr, const float *lead_lam, const float *spt, uint32_t n_scen,
                    const int32_t *bidx, const float *bsc, uint32_t k, int32_t *out_idx, float *out_score,
                    unsigned long long *fl) {
    if (lds && D == 48)
        launch_sweep<K, 48, true, true>(grid, lds_bytes, st, sn, t, rq, hotr, lead_lam, spt, n_scen, bidx, bsc, k,
                                        out_idx, out_score, fl);
    else if (lds && D < 48)
        launch_sweep<K, 48, true, false>(grid, lds_bytes, st, sn, t, rq, hotr, lead_lam, spt, n_scen, bidx, bsc, k,
                                         out_idx, out_score, fl);
    else if (lds)
        launch_sweep<K, 64, true, false>(grid, lds_bytes, st, sn, t, rq, hotr, lead_lam, spt, n_scen, bidx, bsc, k,
                                         out_idx, out_score, fl);
    else
        launch_sweep<K, 64, false, false>(grid, 0, st, sn, t, rq, hotr, lead_lam, spt, n_scen, bidx, bsc, k, out_idx,
                                          out_score, fl);
}

}  // namespace

// ------------------------------------------------------------------ no-allocation scratch
//
// Work buffers of netkv_select_batch_noalloc: one array per device in the
// code object's zero-initialised data, held until the process ends.  In
// host code its name stands for a host-side shadow, not a device address:
// the address on each device is resolved once, with that device current
// (netkv_create), and only that address is used.

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch_dev[kMaxDevices] = {};

// Called with `device` current.
hipError_t resolve_scratch(int device) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[device]) return hipSuccess;
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[device] = (uint8_t *)p;
    return hipSuccess;
}

uint8_t *scratch_of(int device) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_dev[device];
}
}  // namespace

// ------------------------------------------------------------------ API

// ---- for the library's other translation units (netkv_internal.h)

netkv_status netkv_internal_fail(netkv_handle h, netkv_status st, const char *msg) { return fail(h, st, "%s", msg); }

void netkv_internal_clear(netkv_handle h) { h->err.clear(); }

int netkv_internal_device(netkv_handle h) { return h->device; }

uint32_t *netkv_internal_errword(netkv_handle h) { return h->errword; }

hipError_t netkv_internal_flow_buffer(netkv_handle h, uint64_t bytes, void **out) {
    if (bytes > h->flow_buf_bytes) {
        if (h->flow_buf) (void)hipFree(h->flow_buf);
        h->flow_buf = nullptr;
        h->flow_buf_bytes = 0;
        const hipError_t e = hipMalloc(&h->flow_buf, bytes);
        if (e != hipSuccess) return e;
        h->flow_buf_bytes = bytes;
    }
    *out = h->flow_buf;
    return hipSuccess;
}

extern "C" {

netkv_status netkv_create(netkv_handle *out, int device) {
    if (!out) return NETKV_EINVAL;
    *out = nullptr;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return NETKV_EINVAL;
    if (device >= kMaxDevices) return NETKV_EINVAL;
    netkv_handle h = new netkv_ctx();
    h->device = device;
    DeviceGuard g(device);
    if (resolve_scratch(device) != hipSuccess || dalloc(h->errword, 1) != hipSuccess ||
        dalloc(h->loadword, 1) != hipSuccess || hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&h->ev_fork0, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&h->ev_fork1, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&h->ev_inv_fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&h->ev_inv_join, hipEventDisableTiming) != hipSuccess ||
        hipMemset(h->errword, 0, 4) != hipSuccess || hipMemset(h->loadword, 0, 4) != hipSuccess) {
        netkv_destroy(h);
        return NETKV_EDEVICE;
    }
    *out = h;
    return NETKV_OK;
}

void netkv_destroy(netkv_handle h) {
    if (!h) return;
    {
        DeviceGuard g(h->device);
        (void)hipDeviceSynchronize();
        if (h->side) (void)hipStreamDestroy(h->side);
        if (h->flow_buf) (void)hipFree(h->flow_buf);
        if (h->ev_fork0) (void)hipEventDestroy(h->ev_fork0);
        if (h->ev_fork1) (void)hipEventDestroy(h->ev_fork1);
        if (h->ev_join) (void)hipEventDestroy(h->ev_join);
        if (h->ev_inv_fork) (void)hipEventDestroy(h->ev_inv_fork);
        if (h->ev_inv_join) (void)hipEventDestroy(h->ev_inv_join);
        dfree(h->tier_map);
        dfree(h->util);
        dfree(h->n_inflight);
        dfree(h->free_mem);
        dfree(h->queue);
        dfree(h->batch);
        dfree(h->adm_prev);
        dfree(h->sl);
        dfree(h->dbase);
        dfree(h->dxlim);
        dfree(h->table);
        dfree(h->tvals);
        dfree(h->bits);
        dfree(h->errword);
        dfree(h->loadword);
        dfree(h->spt_scen);
        dfree(h->base_idx);
        dfree(h->base_score);
        dfree(h->cnt);
        dfree(h->adm);
        dfree(h->bytes);
        free_scratch(h->sc);
        dfree(h->seq_keys); dfree(h->seq_vals); dfree(h->seq_keys_out); dfree(h->seq_perm);
        dfree(h->seq_start); dfree(h->seq_end);
        for (hipEvent_t ev : h->tev) (void)hipEventDestroy(ev);
        dfree(h->rt1); dfree(h->rt2); dfree(h->ru1); dfree(h->ru2); dfree(h->sr);
    }
    delete h;
}

const char *netkv_last_error(netkv_handle h) { return h ? h->err.c_str() : "NULL handle"; }

netkv_status netkv_oracle_load(netkv_handle h, const netkv_oracle_t *o, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!o) return fail(h, NETKV_EINVAL, "oracle is NULL");
    const uint32_t P = o->n_prefill, D = o->n_decode;
    if (P == 0 || D == 0) return fail(h, NETKV_EINVAL, "n_prefill and n_decode must be >= 1");
    if (D >= (1u << 28) || (uint64_t)P * sl_pitch(D) * 8 >= (1ull << 32))
        return fail(h, NETKV_EINVAL, "n_prefill * (n_decode + 32) must be < 2^29");
    if (!o->tier_map || !o->util || !o->n_inflight || !o->free_mem || !o->queue_depth || !o->batch_size)
        return fail(h, NETKV_EINVAL, "oracle arrays must not be NULL");
    for (int i = 0; i < 4; ++i) {
        if (!(std::isfinite(o->tier_bw[i]) && o->tier_bw[i] > 0.0))
            return fail(h, NETKV_EINVAL, "tier_bw[%d] must be finite and > 0", i);
        if (!finite_nonneg(o->tier_lat[i])) return fail(h, NETKV_EINVAL, "tier_lat[%d] must be >= 0", i);
    }
    if (!finite_nonneg(o->t_iter_a) || !finite_nonneg(o->t_iter_b) || !finite_nonneg(o->alpha))
        return fail(h, NETKV_EINVAL, "t_iter_a, t_iter_b and alpha must be finite and >= 0");
    if (o->block_tokens == 0) return fail(h, NETKV_EINVAL, "block_tokens must be >= 1");
    if (o->kv_bytes_per_token >= (1ull << 32)) return fail(h, NETKV_EINVAL, "kv_bytes_per_token >= 2^32");
    if (h->have_cache && h->cache_D != D)
        return fail(h, NETKV_EINVAL, "snapshot has %u decodes, loaded cache %u", D, h->cache_D);
    DeviceGuard g(h->device);
    hipStream_t st = (hipStream_t)stream;
    const uint64_t npd = (uint64_t)P * D;
    // stage into fresh buffers, validate, then swap in
    uint8_t *tm = nullptr;
    float *ut = nullptr;
    uint16_t *ni = nullptr;
    uint64_t *fm = nullptr, *ap = nullptr;
    uint32_t *qd = nullptr, *bs = nullptr;
    auto cleanup = [&]() {
        dfree(tm); dfree(ut); dfree(ni); dfree(fm); dfree(ap); dfree(qd); dfree(bs);
    };
    if (dalloc(tm, npd) != hipSuccess || dalloc(ut, npd) != hipSuccess || dalloc(ni, 4ull * P) != hipSuccess ||
        dalloc(fm, D) != hipSuccess || dalloc(ap, D) != hipSuccess || dalloc(qd, D) != hipSuccess ||
        dalloc(bs, D) != hipSuccess) {
        cleanup();
        return fail(h, NETKV_ENOMEM, "snapshot allocation failed");
    }
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = hipMemcpyAsync(tm, o->tier_map, npd, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(ut, o->util, npd * 4, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(ni, o->n_inflight, 8ull * P, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(fm, o->free_mem, 8ull * D, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(qd, o->queue_depth, 4ull * D, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(bs, o->batch_size, 4ull * D, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemsetAsync(ap, 0, 8ull * D, st);
    if (e == hipSuccess) e = hipMemsetAsync(h->loadword, 0, 4, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(check_snapshot_kernel, dim3(grid_for(std::max<uint64_t>(npd, D), 256, 4096)), dim3(256),
                           0, st, tm, ut, npd, bs, D, o->beta_max, h->loadword);
        e = hipGetLastError();
    }
    uint32_t bad = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) {
        cleanup();
        return fail(h, NETKV_EDEVICE, "snapshot upload failed: %s", hipGetErrorString(e));
    }
    if (bad) {
        cleanup();
        return fail(h, NETKV_EINVAL, "invalid snapshot:%s%s%s", (bad & 1) ? " tier_map value > 3" : "",
                    (bad & 2) ? " util outside [0,1) or NaN" : "", (bad & 4) ? " batch_size > beta_max" : "");
    }
    if (!h->have_snap || h->P != P || h->D != D) {
        dfree(h->sl); dfree(h->dbase); dfree(h->dxlim);
        // route maps and rows of another shape no longer apply
        dfree(h->rt1); dfree(h->rt2); dfree(h->ru1); dfree(h->ru2); dfree(h->sr);
        h->rt1 = h->rt2 = nullptr;
        h->ru1 = h->ru2 = nullptr;
        h->have_route = false;
        h->have_snap = false;
        if (dalloc(h->sl, (uint64_t)P * sl_pitch(D) + kRowPad) != hipSuccess || dalloc(h->dbase, D) != hipSuccess ||
            dalloc(h->dxlim, D) != hipSuccess) {
            cleanup();
            return fail(h, NETKV_ENOMEM, "snapshot allocation failed");
        }
    }
    dfree(h->tier_map); dfree(h->util); dfree(h->n_inflight); dfree(h->free_mem);
    dfree(h->adm_prev); dfree(h->queue); dfree(h->batch);
    h->tier_map = tm; h->util = ut; h->n_inflight = ni; h->free_mem = fm;
    h->adm_prev = ap; h->queue = qd; h->batch = bs;
    h->P = P;
    h->D = D;
    for (int i = 0; i < 4; ++i) {
        h->bw[i] = (float)o->tier_bw[i];
        h->bw64[i] = o->tier_bw[i];
        h->lat[i] = (float)o->tier_lat[i];
    }
    h->t_a = (float)o->t_iter_a;
    h->t_b = (float)o->t_iter_b;
    h->alpha = (float)o->alpha;
    h->beta_max = o->beta_max;
    h->m_min = o->m_min;
    h->bpt = (uint32_t)o->kv_bytes_per_token;
    h->block_tokens = o->block_tokens;
    h->have_snap = true;
    return NETKV_OK;
}

netkv_status netkv_oracle_set_util(netkv_handle h, const float *util, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    if (!util) return fail(h, NETKV_EINVAL, "util is NULL");
    DeviceGuard g(h->device);
    hipStream_t st = (hipStream_t)stream;
    const uint64_t npd = (uint64_t)h->P * h->D;
    float *ut = nullptr;
    if (dalloc(ut, npd) != hipSuccess) return fail(h, NETKV_ENOMEM, "allocation failed");
    uint32_t bad = 0;
    hipError_t e = hipMemcpyAsync(ut, util, npd * 4, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemsetAsync(h->loadword, 0, 4, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(check_snapshot_kernel, dim3(grid_for(npd, 256, 4096)), dim3(256), 0, st,
                           (const uint8_t *)nullptr, ut, npd, (const uint32_t *)nullptr, 0u, 0u, h->loadword);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess || bad) {
        dfree(ut);
        return e != hipSuccess ? fail(h, NETKV_EDEVICE, "util upload failed: %s", hipGetErrorString(e))
                               : fail(h, NETKV_EINVAL, "invalid util: values outside [0,1) or NaN");
    }
    dfree(h->util);
    h->util = ut;
    return NETKV_OK;
}

netkv_status netkv_congestion_smooth(netkv_handle h, const float *obs, float beta, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    if (!obs) return fail(h, NETKV_EINVAL, "obs is NULL");
    if (!(beta > 0.0f && beta <= 1.0f)) return fail(h, NETKV_EINVAL, "beta must be in (0, 1]");
    DeviceGuard g(h->device);
    hipStream_t st = (hipStream_t)stream;
    const uint64_t npd = (uint64_t)h->P * h->D;
    HIPCHK(h, time_begin(h, st));
    if (((uintptr_t)obs & 15) == 0 && ((uintptr_t)h->util & 15) == 0)
        hipLaunchKernelGGL(smooth_kernel<true>, dim3(grid_for((npd + 3) / 4, 256, 8192)), dim3(256), 0, st, h->util,
                           obs, npd, beta, h->errword);
    else
        hipLaunchKernelGGL(smooth_kernel<false>, dim3(grid_for(npd, 256, 8192)), dim3(256), 0, st, h->util, obs,
                           npd, beta, h->errword);
    HIPCHK(h, hipGetLastError());
    HIPCHK(h, time_end(h, st));
    return NETKV_OK;
}

netkv_status netkv_congestion_get(netkv_handle h, float *out, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    if (!out) return fail(h, NETKV_EINVAL, "out is NULL");
    DeviceGuard g(h->device);
    HIPCHK(h, hipMemcpyAsync(out, h->util, (uint64_t)h->P * h->D * sizeof(float), hipMemcpyDeviceToDevice,
                             (hipStream_t)stream));
    return NETKV_OK;
}

netkv_status netkv_route2_load(netkv_handle h, const uint8_t *tier1, const float *util1, const uint8_t *tier2,
                               const float *util2, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    if (!tier1 || !util1 || !tier2 || !util2) return fail(h, NETKV_EINVAL, "a route map is NULL");
    DeviceGuard g(h->device);
    hipStream_t st = (hipStream_t)stream;
    const uint64_t npd = (uint64_t)h->P * h->D;
    uint8_t *a = nullptr, *b = nullptr;
    float *ua = nullptr, *ub = nullptr;
    auto drop = [&]() { dfree(a); dfree(b); dfree(ua); dfree(ub); };
    if (dalloc(a, npd) != hipSuccess || dalloc(b, npd) != hipSuccess || dalloc(ua, npd) != hipSuccess ||
        dalloc(ub, npd) != hipSuccess || (!h->sr && dalloc(h->sr, (uint64_t)h->P * sl_pitch(h->D) + kRowPad) != hipSuccess)) {
        drop();
        return fail(h, NETKV_ENOMEM, "route map allocation failed");
    }
    uint32_t bad = 0;
    hipError_t e = hipMemcpyAsync(a, tier1, npd, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(b, tier2, npd, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(ua, util1, npd * 4, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(ub, util2, npd * 4, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemsetAsync(h->loadword, 0, 4, st);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(check_snapshot_kernel, dim3(grid_for(npd, 256, 4096)), dim3(256), 0, st,
                           (const uint8_t *)a, (const float *)ua, npd, (const uint32_t *)nullptr, 0u, 0u,
                           h->loadword);
        hipLaunchKernelGGL(check_snapshot_kernel, dim3(grid_for(npd, 256, 4096)), dim3(256), 0, st,
                           (const uint8_t *)b, (const float *)ub, npd, (const uint32_t *)nullptr, 0u, 0u,
                           h->loadword);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess || bad) {
        drop();
        return e != hipSuccess ? fail(h, NETKV_EDEVICE, "route map upload failed: %s", hipGetErrorString(e))
                               : fail(h, NETKV_EINVAL, "invalid route map:%s%s", (bad & 1) ? " tier value > 3" : "",
                                      (bad & 2) ? " util outside [0,1) or NaN" : "");
    }
    dfree(h->rt1);
    dfree(h->rt2);
    dfree(h->ru1);
    dfree(h->ru2);
    h->rt1 = a;
    h->rt2 = b;
    h->ru1 = ua;
    h->ru2 = ub;
    h->have_route = true;
    return NETKV_OK;
}

netkv_status netkv_route2_clear(netkv_handle h) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    DeviceGuard g(h->device);
    dfree(h->rt1);
    dfree(h->rt2);
    dfree(h->ru1);
    dfree(h->ru2);
    h->rt1 = h->rt2 = nullptr;
    h->ru1 = h->ru2 = nullptr;
    h->have_route = false;
    return NETKV_OK;
}

netkv_status netkv_route2_of(netkv_handle h, const netkv_requests_t *req, uint32_t k, const int32_t *idx,
                             int8_t *out_route, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (req->n_req && (!idx || !out_route)) return fail(h, NETKV_EINVAL, "idx and out_route must not be NULL");
    if ((st = ready(h))) return st;
    if (!h->have_route) return fail(h, NETKV_ENOTREADY, "no route maps loaded (netkv_route2_load)");
    if (req->n_req == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    Snap sn = make_snap(h);
    const uint64_t nd = std::max<uint64_t>((uint64_t)h->P * h->D, h->D);
    hipLaunchKernelGGL(derive_kernel, dim3((uint32_t)((nd + 255) / 256)), dim3(256), 0, s, sn, h->sl, h->dbase,
                       h->dxlim);
    hipLaunchKernelGGL(derive_route_kernel, dim3((uint32_t)((nd + 255) / 256)), dim3(256), 0, s, sn,
                       (const uint8_t *)h->rt1, (const float *)h->ru1, (const uint8_t *)h->rt2,
                       (const float *)h->ru2, h->sr);
    sn.sr = h->sr;
    const uint64_t n = (uint64_t)req->n_req * k;
    hipLaunchKernelGGL(route_of_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, sn, make_table(h),
                       make_reqs(req), k, idx, out_route);
    HIPCHK(h, hipGetLastError());
    return NETKV_OK;
}

netkv_status netkv_selection_bytes(netkv_handle h, const netkv_requests_t *req, uint32_t k, const int32_t *idx,
                                   uint64_t *out_bytes, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (req->n_req && (!idx || !out_bytes)) return fail(h, NETKV_EINVAL, "idx and out_bytes must not be NULL");
    if ((st = ready(h))) return st;
    if (req->n_req == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    const uint64_t n = (uint64_t)req->n_req * k;
    hipLaunchKernelGGL(selection_bytes_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                       make_snap(h), make_table(h), make_reqs(req), k, idx, out_bytes, h->errword);
    HIPCHK(h, hipGetLastError());
    return NETKV_OK;
}

netkv_status netkv_cache_load(netkv_handle h, uint32_t n_decode, const uint64_t *hash_off, const uint64_t *hashes,
                              uint64_t n_hashes, float max_load_factor, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (n_decode == 0 || !hash_off) return fail(h, NETKV_EINVAL, "n_decode must be >= 1 and hash_off non-NULL");
    if (n_hashes && !hashes) return fail(h, NETKV_EINVAL, "hashes is NULL");
    if (!(max_load_factor > 0.0f && max_load_factor < 1.0f))
        return fail(h, NETKV_EINVAL, "max_load_factor must be in (0, 1)");
    if (h->have_snap && h->D != n_decode)
        return fail(h, NETKV_EINVAL, "cache has %u decodes, loaded snapshot %u", n_decode, h->D);
    DeviceGuard g(h->device);
    hipStream_t st = (hipStream_t)stream;
    std::vector<uint64_t> off(n_decode + 1);
    HIPCHK(h, hipMemcpyAsync(off.data(), hash_off, 8ull * (n_decode + 1), hipMemcpyDefault, st));
    HIPCHK(h, hipStreamSynchronize(st));
    for (uint32_t d = 0; d < n_decode; ++d)
        if (off[d + 1] < off[d]) return fail(h, NETKV_EINVAL, "hash_off decreases at decode %u", d);
    if (off[n_decode] > n_hashes) return fail(h, NETKV_EINVAL, "hash_off[n_decode] exceeds n_hashes");
    const uint64_t first = off[0], total = off[n_decode] - off[0];
    if (total >= (1ull << 31)) return fail(h, NETKV_ECAPACITY, "more than 2^31 - 1 resident hashes");
    // words per holder bitmap row: whole 64-decode words, rounded up to a
    // multiple of 12 so that every decodes-per-lane choice C (1, 2, 3, 4, 6)
    // reads its groups' C words inside the row, at 8 * C-byte alignment
    const uint64_t bwords = ((uint64_t)n_decode + 63) / 64;
    const uint32_t bpitch = (uint32_t)((bwords + 11) / 12 * 12);
    uint64_t *dh = nullptr, *dkey = nullptr, *doff = nullptr;
    uint32_t *dec_in = nullptr, *dec = nullptr;
    unsigned long long *cnt = nullptr;
    uint8_t *stmp = nullptr;
    auto cleanup = [&]() { dfree(dh); dfree(dkey); dfree(doff); dfree(dec_in); dfree(dec); dfree(cnt); dfree(stmp); };
    // the device copy keeps the caller's absolute offsets valid: copy from `first`
    if (dalloc(dh, off[n_decode]) != hipSuccess || dalloc(doff, (uint64_t)n_decode + 1) != hipSuccess ||
        dalloc(dkey, total) != hipSuccess || dalloc(dec_in, total) != hipSuccess ||
        dalloc(dec, total) != hipSuccess || dalloc(cnt, 2) != hipSuccess) {
        cleanup();
        return fail(h, NETKV_ENOMEM, "staging allocation failed");
    }
    hipError_t e = hipSuccess;
    if (total) e = hipMemcpyAsync(dh + first, hashes + first, 8ull * total, hipMemcpyDefault, st);
    if (e == hipSuccess) e = hipMemcpyAsync(doff, off.data(), 8ull * (n_decode + 1), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipMemsetAsync(h->loadword, 0, 4, st);
    uint32_t bad = 0;
    if (e == hipSuccess && total) {
        hipLaunchKernelGGL(count_zero_kernel, dim3(grid_for(total, 256, 8192)), dim3(256), 0, st, dh + first, total,
                           h->loadword);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) {
        cleanup();
        return fail(h, NETKV_EDEVICE, "cache upload failed: %s", hipGetErrorString(e));
    }
    if (bad) {
        cleanup();
        return fail(h, NETKV_EINVAL, "cache contains the reserved hash value 0");
    }
    // (hash, decode) pairs sorted by hash; per distinct hash: one holder or several
    unsigned long long counts[2] = {0, 0};
    if (total) {
        hipLaunchKernelGGL(owner_kernel, dim3(grid_for(total, 256, 16384)), dim3(256), 0, st, (const uint64_t *)doff,
                           n_decode, first, total, dec_in);
        e = hipGetLastError();
        size_t tb = 0;
        if (e == hipSuccess)
            e = rocprim::radix_sort_pairs(nullptr, tb, (const uint64_t *)(dh + first), dkey, (const uint32_t *)dec_in,
                                          dec, (uint32_t)total, 0, 64, st);
        if (e == hipSuccess && dalloc(stmp, std::max<size_t>(tb, 16)) != hipSuccess) {
            cleanup();
            return fail(h, NETKV_ENOMEM, "sort scratch allocation failed");
        }
        if (e == hipSuccess)
            e = rocprim::radix_sort_pairs(stmp, tb, (const uint64_t *)(dh + first), dkey, (const uint32_t *)dec_in,
                                          dec, (uint32_t)total, 0, 64, st);
        if (e == hipSuccess) e = hipMemsetAsync(cnt, 0, 16, st);
        if (e == hipSuccess) {
            hipLaunchKernelGGL(classify_kernel, dim3(grid_for(total, 256, 16384)), dim3(256), 0, st,
                               (const uint64_t *)dkey, (const uint32_t *)dec, total, cnt);
            e = hipGetLastError();
        }
        if (e == hipSuccess) e = hipMemcpyAsync(counts, cnt, 16, hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
    }
    dfree(dh);
    dfree(doff);
    dfree(dec_in);
    dfree(stmp);
    if (e != hipSuccess) {
        cleanup();
        return fail(h, NETKV_EDEVICE, "holder sort failed: %s", hipGetErrorString(e));
    }
    const uint64_t distinct = counts[0], rows = counts[1] + 1;   // row 0: all zero
    if (rows >= (uint64_t)kHeldOne) {
        cleanup();
        return fail(h, NETKV_ECAPACITY, "more than 2^31 - 2 hashes held by several decodes");
    }
    // release the old index first: the new one may be large
    dfree(h->table);
    dfree(h->tvals);
    dfree(h->bits);
    h->have_cache = false;
    // two slots per bucket; two-choice cuckoo sets of 2-slot buckets stay
    // buildable well above load factor 0.5, and are capped at 0.85
    const double lf = std::min(0.85, (double)max_load_factor);
    const uint64_t need = (uint64_t)std::ceil((double)distinct / (2.0 * lf));
    uint32_t log2b = 3;
    while ((1ull << log2b) < need) {
        ++log2b;
        if (log2b > 30) {
            cleanup();
            return fail(h, NETKV_ECAPACITY, "the index would need more than 2^31 slots");
        }
    }
    uint64_t *tab = nullptr, *bm = nullptr;
    uint32_t *tv = nullptr;
    if (dalloc(bm, rows * bpitch) != hipSuccess) {
        cleanup();
        return fail(h, NETKV_ENOMEM, "holder bitmap allocation of %llu bytes failed",
                    (unsigned long long)(8 * rows * bpitch));
    }
    e = hipMemsetAsync(bm, 0, 8 * rows * bpitch, st);
    // build at the planned size; should a build fail to place every key (a
    // random walk that did not end), rebuild with twice the buckets, twice
    uint64_t nbk = 0;
    for (int attempt = 0;; ++attempt) {
        nbk = 1ull << log2b;
        if (e == hipSuccess && (dalloc(tab, 2 * nbk) != hipSuccess || dalloc(tv, 2 * nbk) != hipSuccess)) {
            cleanup();
            dfree(tab); dfree(tv); dfree(bm);
            return fail(h, NETKV_ENOMEM, "index allocation of %llu bytes failed", (unsigned long long)(24 * nbk));
        }
        if (e == hipSuccess) e = hipMemsetAsync(tab, 0, 16 * nbk, st);
        if (e == hipSuccess) e = hipMemsetAsync(h->loadword, 0, 4, st);
        if (e == hipSuccess && total) {
            hipLaunchKernelGGL(index_insert_kernel, dim3(grid_for(total, 256, 16384)), dim3(256), 0, st, tab,
                               64u - log2b, (const uint64_t *)dkey, total, h->loadword);
            e = hipGetLastError();
        }
        bad = 0;
        if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess || !bad || attempt == 2 || log2b >= 30) break;
        dfree(tab);
        dfree(tv);
        ++log2b;
    }
    if (e == hipSuccess && !bad && total) {
        // rows are handed out from 1 (cnt[0] doubles as the counter)
        const uint32_t one = 1;
        e = hipMemcpyAsync(cnt, &one, 4, hipMemcpyHostToDevice, st);
        if (e == hipSuccess) {
            hipLaunchKernelGGL(index_value_kernel, dim3(grid_for(total, 256, 16384)), dim3(256), 0, st,
                               (const uint64_t *)tab, tv, 64u - log2b, bm, bpitch, (const uint64_t *)dkey,
                               (const uint32_t *)dec, total, (uint32_t *)cnt, h->loadword);
            e = hipGetLastError();
        }
        if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
    }
    cleanup();
    if (e != hipSuccess || bad) {
        dfree(tab);
        dfree(tv);
        dfree(bm);
        return e != hipSuccess ? fail(h, NETKV_EDEVICE, "index build failed: %s", hipGetErrorString(e))
                               : fail(h, NETKV_ECAPACITY, "index build could not place every hash");
    }
    h->table = tab;
    h->tvals = tv;
    h->bits = bm;
    h->buckets = nbk;
    h->log2b = log2b;
    h->bpitch = bpitch;
    h->rows = rows;
    h->distinct = distinct;
    h->table_bytes = 24 * nbk + 8 * rows * bpitch;
    h->cache_D = n_decode;
    h->have_cache = true;
    return NETKV_OK;
}

netkv_status netkv_select_batch(netkv_handle h, const netkv_requests_t *req, uint32_t k, int32_t *out_idx,
                                float *out_score, netkv_pairs_t *pairs, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (req->n_req && (!out_idx || !out_score))
        return fail(h, NETKV_EINVAL, "out_idx and out_score must not be NULL");
    if ((st = ready(h))) return st;
    if (req->n_req == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    PairOut po{nullptr, nullptr, nullptr};
    bool want_pairs = false;
    if (pairs) {
        po.j = pairs->prefix_blocks;
        po.feas = pairs->feasible;
        po.score = pairs->score;
        want_pairs = po.j || po.feas || po.score;
    }
    return select_owned(h, req, k, out_idx, out_score, po, want_pairs, 0xFFFFFFFFu, s, true);
}

netkv_status netkv_select_batch_noalloc(netkv_handle h, const netkv_requests_t *req, uint32_t k, int32_t *out_idx,
                                        float *out_score, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (req->n_req && (!out_idx || !out_score))
        return fail(h, NETKV_EINVAL, "out_idx and out_score must not be NULL");
    if ((st = ready(h))) return st;
    if (req->n_req == 0) return NETKV_OK;
    uint8_t *base = scratch_of(h->device);
    if (!base) return fail(h, NETKV_EDEVICE, "no-allocation scratch not resolved on device %d", h->device);
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    Scratch sc;
    uint64_t r_sub = 0;
    if ((st = carve_static(h, base, req->n_req, k, sc, r_sub))) return st;
    const PairOut po{nullptr, nullptr, nullptr};
    for (uint64_t r0 = 0; r0 < req->n_req; r0 += r_sub) {
        netkv_requests_t sub = *req;
        sub.n_req = (uint32_t)std::min<uint64_t>(r_sub, req->n_req - r0);
        sub.prefill += r0;
        sub.len_tokens += r0;
        sub.hash_off += r0;   // absolute offsets into the same hash array
        if ((st = run_select(h, sc, &sub, k, out_idx + r0 * k, out_score + r0 * k, po, false, 0xFFFFFFFFu, s, true,
                             r0 == 0)))
            return st;
    }
    return NETKV_OK;
}

netkv_status netkv_reserve(netkv_handle h, uint32_t max_req, uint64_t max_hashes, uint32_t max_k, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (max_k < 1 || max_k > 8) return fail(h, NETKV_EINVAL, "max_k must be in [1, 8]");
    if (max_req > (1u << 31)) return fail(h, NETKV_EINVAL, "max_req too large");
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded (netkv_oracle_load)");
    if (max_req == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    uint64_t elems = 0;
    for (uint32_t k = 1; k <= max_k; ++k) {
        const Geometry geo = geometry(h, k);
        elems = std::max<uint64_t>(elems, (uint64_t)max_req * geo.ngroup * geo.K);
    }
    netkv_status st = ensure_scratch(h, h->sc, max_req, elems, max_hashes, (hipStream_t)stream);
    if (!st) st = ensure_hotr(h, max_req);
    if (!st) st = ensure_seq(h, max_req, h->P, true, true);
    return st;
}

netkv_status netkv_rank_sweep(netkv_handle h, const netkv_requests_t *req, uint32_t n_scen, const float *util_scen,
                              uint32_t k, int32_t *out_idx, float *out_score, uint64_t *out_flips,
                              uint64_t *out_inversions, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (n_scen > 65535) return fail(h, NETKV_EINVAL, "n_scen must be <= 65535");
    if (n_scen && !util_scen) return fail(h, NETKV_EINVAL, "util_scen must not be NULL");
    if (n_scen && req->n_req && (!out_idx || !out_score))
        return fail(h, NETKV_EINVAL, "out_idx and out_score must not be NULL");
    if ((st = ready(h))) return st;
    if (n_scen == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    const uint64_t R = req->n_req, P = h->P, D = h->D;
    Snap sn = make_snap(h);
    if (out_flips) {
        hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(2ull * n_scen, 256)), dim3(256), 0, s, out_flips,
                           2ull * n_scen, 0ull);
        HIPCHK(h, hipGetLastError());
    }
    // The caller's stream waits for the second stream when the call
    // returns (every path), if the counts below were forked onto it.
    struct Join {
        hipStream_t s;
        hipEvent_t e;
        bool on = false;
        ~Join() {
            if (on) (void)hipStreamWaitEvent(s, e, 0);
        }
    } join{s, h->ev_inv_join};
    if (out_inversions) {
        // Proposition 2's counts depend on the snapshot and the scenarios
        // only.  When the selection below leaves the second stream free (a
        // batch below kForkMinN requests) they run there, beside the
        // selection and the sweep.
        const bool fork = R > 0 && R < kForkMinN;
        hipStream_t si = fork ? h->side : s;
        if (fork) {
            HIPCHK(h, hipEventRecord(h->ev_inv_fork, s));
            HIPCHK(h, hipStreamWaitEvent(si, h->ev_inv_fork, 0));
        }
        hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(3ull * n_scen, 256)), dim3(256), 0, si, out_inversions,
                           3ull * n_scen, 0ull);
        Bw64 bw;
        for (int i = 0; i < 4; ++i) bw.b[i] = h->bw64[i];
        hipLaunchKernelGGL(tier_inv_kernel, dim3((uint32_t)((P * D + 255) / 256), n_scen), dim3(256), 0, si, sn, bw,
                           util_scen, (unsigned long long *)out_inversions);
        HIPCHK(h, hipGetLastError());
        if (fork) {
            HIPCHK(h, hipEventRecord(h->ev_inv_join, si));
            join.on = true;
        }
    }
    if (R == 0) return NETKV_OK;
    if ((st = ensure_seq(h, R, P, false, true))) return st;
    const uint64_t nspt = (uint64_t)n_scen * P * D;
    if (h->spt_cap < nspt) {
        dfree(h->spt_scen);
        h->spt_cap = 0;
        HIPCHK(h, dalloc(h->spt_scen, nspt));
        h->spt_cap = nspt;
    }
    // the selection under the loaded congestion, keeping every request's
    // scoring record by batch index and the leaders' prefix lengths
    {
        TimingOff off(h);  // only the sweep kernel is timed
        const PairOut po{nullptr, nullptr, nullptr};
        if ((st = select_owned(h, req, 1, h->base_idx, h->base_score, po, false, 0xFFFFFFFFu, s, false, true)))
            return st;
    }
    hipLaunchKernelGGL(derive_scen_kernel, dim3((uint32_t)((nspt + 255) / 256)), dim3(256), 0, s, sn, util_scen, nspt,
                       h->spt_scen);
    HIPCHK(h, hipGetLastError());
    const Reqs rq = make_reqs(req);
    const Table t = make_table(h);
    const uint32_t Dp = (uint32_t)D | 1u;
    const bool lds = P * Dp <= kSweepMaxTab;
    // a third table (the next scenario's) when the threads hold its entries
    const bool held = (uint64_t)P * D <= (uint64_t)kSweepThreads * kSweepHold;
    const size_t lds_bytes = lds ? (held ? 3 : 2) * P * Dp * sizeof(float) : 0;
    const dim3 grid((uint32_t)((R + kSweepThreads - 1) / kSweepThreads), (n_scen + kSweepScen - 1) / kSweepScen);
    unsigned long long *fl = (unsigned long long *)out_flips;
    HIPCHK(h, time_begin(h, s));
#define NETKV_SWEEP(KK)                                                                                            \
    launch_sweep_k<KK>((uint32_t)D, lds, grid, lds_bytes, s, sn, t, rq, h->sc.hotr, h->sc.lead_lam, h->spt_scen,    \
                       n_scen, h->base_idx, h->base_score, k, out_idx, out_score, fl)
    if (k == 1) NETKV_SWEEP(1);
    else if (k == 2) NETKV_SWEEP(2);
    else if (k == 3) NETKV_SWEEP(3);
    else if (k == 4) NETKV_SWEEP(4);
    else NETKV_SWEEP(8);
#undef NETKV_SWEEP
    HIPCHK(h, hipGetLastError());
    HIPCHK(h, time_end(h, s));
    return NETKV_OK;
}

netkv_status netkv_commit_batch(netkv_handle h, const netkv_requests_t *req, const int32_t *sel, uint32_t cap,
                                uint32_t mu, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (!sel && req->n_req) return fail(h, NETKV_EINVAL, "sel is NULL");
    if (cap > 65535) return fail(h, NETKV_EINVAL, "cap must be <= 65535");
    if ((st = ready(h))) return st;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    if (h->commit_P != h->P || h->commit_D != h->D) {
        dfree(h->cnt);
        dfree(h->adm);
        dfree(h->bytes);
        h->commit_P = h->commit_D = 0;
        HIPCHK(h, dalloc(h->cnt, 4ull * h->P));
        HIPCHK(h, dalloc(h->adm, h->D));
        HIPCHK(h, dalloc(h->bytes, h->D));
        h->commit_P = h->P;
        h->commit_D = h->D;
    }
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(4ull * h->P, 256)), dim3(256), 0, s, h->cnt, 4ull * h->P, 0u);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(h->D, 256)), dim3(256), 0, s, h->adm, (uint64_t)h->D, 0u);
    hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(h->D, 256)), dim3(256), 0, s, (uint64_t *)h->bytes,
                       (uint64_t)h->D, 0ull);
    HIPCHK(h, hipGetLastError());
    if (req->n_req) {
        hipLaunchKernelGGL(commit_count_kernel, dim3((req->n_req + 255) / 256), dim3(256), 0, s, make_snap(h),
                           make_table(h), make_reqs(req), sel, h->cnt, h->adm, h->bytes, h->errword);
        HIPCHK(h, hipGetLastError());
    }
    uint32_t n = std::max(4u * h->P, h->D);
    hipLaunchKernelGGL(commit_apply_kernel, dim3((n + 255) / 256), dim3(256), 0, s, h->P, h->D, cap, mu,
                       (const uint32_t *)h->cnt, (const uint32_t *)h->adm, (const unsigned long long *)h->bytes,
                       h->n_inflight, h->queue, h->free_mem, h->adm_prev);
    HIPCHK(h, hipGetLastError());
    return NETKV_OK;
}

netkv_status netkv_state_get(netkv_handle h, uint16_t *n_inflight, uint32_t *queue_depth, uint64_t *free_mem,
                             uint64_t *admitted_prev, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    if (n_inflight) HIPCHK(h, hipMemcpyAsync(n_inflight, h->n_inflight, 8ull * h->P, hipMemcpyDefault, s));
    if (queue_depth) HIPCHK(h, hipMemcpyAsync(queue_depth, h->queue, 4ull * h->D, hipMemcpyDefault, s));
    if (free_mem) HIPCHK(h, hipMemcpyAsync(free_mem, h->free_mem, 8ull * h->D, hipMemcpyDefault, s));
    if (admitted_prev) HIPCHK(h, hipMemcpyAsync(admitted_prev, h->adm_prev, 8ull * h->D, hipMemcpyDefault, s));
    HIPCHK(h, hipStreamSynchronize(s));
    return NETKV_OK;
}

netkv_status netkv_sync_errors(netkv_handle h, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    uint32_t e = 0;
    HIPCHK(h, hipStreamSynchronize(s));
    HIPCHK(h, hipMemcpy(&e, h->errword, 4, hipMemcpyDeviceToHost));
    HIPCHK(h, hipMemset(h->errword, 0, 4));
    if (e)
        return fail(h, NETKV_EINVAL, "input errors:%s%s%s%s%s%s",
                    (e & kErrRequest) ? " inconsistent request header" : "",
                    (e & kErrObservation) ? " congestion observation outside [0,1)" : "",
                    (e & kErrSelection) ? " selection index >= D" : "", (e & kErrTableFull) ? " table full" : "",
                    (e & kErrFlow) ? " invalid flow set" : "",
                    (e & kErrFlowStall) ? " flow simulation reached its iteration bound" : "");
    return NETKV_OK;
}

netkv_status netkv_set_timing(netkv_handle h, int enable) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (enable && h->tev.empty()) {
        DeviceGuard g(h->device);
        h->tev.assign(2 * kTimeSlots, nullptr);
        for (hipEvent_t &ev : h->tev) HIPCHK(h, hipEventCreate(&ev));
    }
    h->timing = enable != 0;
    h->tcount = 0;
    return NETKV_OK;
}

netkv_status netkv_kernel_ms(netkv_handle h, float *ms) {
    if (!h || !ms) return NETKV_EINVAL;
    h->err.clear();
    if (h->tcount == 0) return fail(h, NETKV_ENOTREADY, "no timed kernel yet");
    DeviceGuard g(h->device);
    const uint32_t n = std::min(h->tcount, kTimeSlots);
    const uint32_t last = (h->tcount - 1) % kTimeSlots;
    HIPCHK(h, hipEventSynchronize(h->tev[2 * last + 1]));
    double sum = 0.0;
    for (uint32_t i = 0; i < n; ++i) {
        const uint32_t slot = (h->tcount - 1 - i) % kTimeSlots;
        float one = 0.0f;
        HIPCHK(h, hipEventElapsedTime(&one, h->tev[2 * slot], h->tev[2 * slot + 1]));
        sum += one;
    }
    *ms = (float)(sum / n);
    return NETKV_OK;
}

netkv_status netkv_tier_counts(netkv_handle h, const netkv_requests_t *req, const int32_t *sel, uint64_t *counts,
                               void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (!counts || (req->n_req && !sel)) return fail(h, NETKV_EINVAL, "sel and counts must not be NULL");
    if (!h->have_snap) return fail(h, NETKV_ENOTREADY, "no snapshot loaded");
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    hipLaunchKernelGGL(fill_u64_kernel, dim3(1), dim3(64), 0, s, counts, (uint64_t)5, 0ull);
    if (req->n_req)
        hipLaunchKernelGGL(tier_count_kernel, dim3((req->n_req + 255) / 256), dim3(256), 0, s, make_snap(h),
                           make_reqs(req), sel, (unsigned long long *)counts, h->errword);
    HIPCHK(h, hipGetLastError());
    return NETKV_OK;
}

netkv_status netkv_select_sequential(netkv_handle h, const netkv_requests_t *req, uint32_t cap, int32_t *out_idx,
                                     float *out_score, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (req->n_req && (!out_idx || !out_score)) return fail(h, NETKV_EINVAL, "out_idx and out_score must not be NULL");
    if (cap > 65535) return fail(h, NETKV_EINVAL, "cap must be <= 65535");
    if ((st = ready(h))) return st;
    if (req->n_req == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    const uint64_t R = req->n_req, P = h->P;
    if ((st = ensure_seq(h, R, P, true, false))) return st;
    // validation, every request's scoring record by batch index and the
    // leaders' prefix lengths, by the batch selection (its outputs are then
    // overwritten by the chain; invalid requests keep -1 / NaN)
    {
        TimingOff off(h);  // only the sequential kernel is timed
        const PairOut po{nullptr, nullptr, nullptr};
        if ((st = select_owned(h, req, 1, out_idx, out_score, po, false, 0xFFFFFFFFu, s, false, true))) return st;
    }
    // requests grouped by prefill instance, batch order kept inside a group
    const Reqs rq = make_reqs(req);
    hipLaunchKernelGGL(prefill_key_kernel, dim3((uint32_t)((R + 255) / 256)), dim3(256), 0, s, rq, (uint32_t)P,
                       (const uint32_t *)h->sc.keys_in, h->seq_keys, h->seq_vals);
    size_t tb = h->sc.sort_tmp_bytes;
    if (R > kSortMinN && R <= kSortMaxN && h->sc.sort_cnt)
        HIPCHK(h, batch_sort_pairs(h, h->sc, h->seq_keys, h->seq_vals, h->seq_keys_out, h->seq_perm, (uint32_t)R,
                                   bits_for(P), s));
    else
        HIPCHK(h, rocprim::radix_sort_pairs<SortConfig>(h->sc.sort_tmp, tb, h->seq_keys, h->seq_keys_out,
                                                        h->seq_vals, h->seq_perm, (uint32_t)R, 0, bits_for(P), s));
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(P, 256)), dim3(256), 0, s, h->seq_start, P, 0u);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(P, 256)), dim3(256), 0, s, h->seq_end, P, 0u);
    hipLaunchKernelGGL(segment_kernel, dim3((uint32_t)((R + 255) / 256)), dim3(256), 0, s,
                       (const uint32_t *)h->seq_keys_out, (uint32_t)R, (uint32_t)P, h->seq_start, h->seq_end);
    HIPCHK(h, hipGetLastError());
    HIPCHK(h, time_begin(h, s));
    const Snap sn = make_snap(h);
    const Table t = make_table(h);
    const Hot *hr = h->sc.hotr;
    const float *ll = h->sc.lead_lam;
    const uint32_t *ord = h->seq_perm, *b0 = h->seq_start, *b1 = h->seq_end;
    // one workgroup per prefill instance, all of them resident at once on
    // 256 CUs up to 1,024 prefills (256 threads: four workgroups per CU
    // within the register budget); a thread holds MAXC decodes
#define NETKV_SEQ(TT, MC)                                                                                       \
    hipLaunchKernelGGL((sequential_cached_kernel<TT, MC>), dim3((uint32_t)P), dim3(TT), 0, s, sn, t, rq, cap, hr, ll, \
                       ord, b0, b1, out_idx, out_score)
    const uint32_t Dn = h->D;
    if (Dn <= 64) NETKV_SEQ(64, 1);
    else if (Dn <= 256) NETKV_SEQ(256, 1);
    else if (Dn <= 512) NETKV_SEQ(256, 2);
    else if (Dn <= 1024) NETKV_SEQ(256, 4);
    else if (Dn <= 1536) NETKV_SEQ(256, 6);
    else if (Dn <= 2048) NETKV_SEQ(256, 8);
    else if (Dn <= 3072) NETKV_SEQ(256, 12);
    else if (Dn <= 4096) NETKV_SEQ(256, 16);
    else
        hipLaunchKernelGGL(sequential_kernel, dim3((uint32_t)P), dim3(kSeqThreads), 0, s, sn, t, rq, cap, hr, ll, ord,
                           b0, b1, out_idx, out_score);
#undef NETKV_SEQ
    HIPCHK(h, hipGetLastError());
    HIPCHK(h, time_end(h, s));
    return NETKV_OK;
}

netkv_status netkv_set_option(netkv_handle h, int option, uint32_t value) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    switch (option) {
    case NETKV_OPT_RUN_LEN:
        if (value > (1u << 20)) return fail(h, NETKV_EINVAL, "run length must be <= 2^20");
        h->run_len_opt = value;
        return NETKV_OK;
    case NETKV_OPT_REUSE:
        h->reuse_opt = value ? 1u : 0u;
        return NETKV_OK;
    case NETKV_OPT_POLICY:
        if (value > 2) return fail(h, NETKV_EINVAL, "policy must be 0 (full), 1 (no congestion) or 2 (topology only)");
        h->policy_opt = value;
        return NETKV_OK;
    case NETKV_OPT_LEAD_CAP:
        h->lead_cap_opt = value;
        return NETKV_OK;
    case NETKV_OPT_COLS:
        if (value != 0 && value != 1 && value != 2 && value != 3 && value != 4 && value != 6)
            return fail(h, NETKV_EINVAL, "decodes per lane must be 0 (automatic), 1, 2, 3, 4 or 6");
        h->cols_opt = value;
        return NETKV_OK;
    default:
        return fail(h, NETKV_EINVAL, "unknown option %d", option);
    }
}

netkv_status netkv_cache_info(netkv_handle h, uint64_t *index_slots, uint64_t *distinct_hashes,
                              uint64_t *shared_hashes, uint64_t *index_bytes) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    if (!h->have_cache) return fail(h, NETKV_ENOTREADY, "no cache loaded (netkv_cache_load)");
    if (index_slots) *index_slots = 2 * h->buckets;
    if (distinct_hashes) *distinct_hashes = h->distinct;
    if (shared_hashes) *shared_hashes = h->rows - 1;
    if (index_bytes) *index_bytes = h->table_bytes;
    return NETKV_OK;
}

}  // extern "C"

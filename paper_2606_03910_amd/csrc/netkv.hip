// libnetkv -- NetKV decode-instance selection for MI355X (gfx950).
//
// Host runtime and HIP kernels behind the C ABI declared in include/netkv.h.
// Method: "NetKV: Network-Aware Decode Instance Selection for Disaggregated
// LLM Inference", Algorithm 1 with Eqs. (2)-(7), evaluated for a whole batch
// of requests against one telemetry snapshot.
//
// Data layout in device memory (all owned by the handle):
//   * resident-set tables: one open-addressed table per decode, all with the
//     same power-of-two capacity and the same slot function, stored
//     slot-major: table[slot * pitch + d] (pitch = D rounded up to 16).
//     A wavefront scoring one request against 64 consecutive decodes probes
//     the same slot index in all 64 tables, so each probe step is one
//     contiguous 512-byte row segment: fully coalesced, whatever the hash.
//     Empty slots hold 0 (hash value 0 is reserved).  Linear probing.
//   * snapshot: tier_map u8[P*D], util f32[P*D] (row-major by prefill),
//     n_inflight u16[4*P] (tier-major), free_mem u64[D], queue u32[D],
//     batch u32[D], plus the admitted bytes of the previous batch u64[D].
//
// Kernels:
//   select_kernel  -- prefix match (Sec. III-B) + Eqs. (2)-(7) + feasibility
//                     + per-request top-k, fused; one wavefront per request,
//                     lanes over decodes; optional per-pair outputs.
//   sweep_kernel   -- re-scoring under congestion scenarios with the prefix
//                     lengths reused; lanes over requests.
//   insert_kernel  -- builds the tables with 64-bit compare-and-swap.
//   commit kernels -- between-batch counter / queue / memory update.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "netkv.h"

namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kStage = 256;           // hashes of one request staged in LDS
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kEmptyKey = ~0ull; // empty top-k entry (sorts last)

enum : uint32_t {
    kErrRequest = 1u,    // request header inconsistent
    kErrZeroHash = 2u,   // request carries hash 0
    kErrSelection = 4u,  // selection index out of range
    kErrTableFull = 8u,  // insertion found no free slot
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
};

struct Table {
    const uint64_t *keys;
    uint64_t mask;
    uint32_t shift;   // 64 - log2(capacity)
    uint32_t pitch;
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
    uint16_t *jT;       // [D][R] (internal, for the sweep)
};

__host__ __device__ inline uint64_t home_slot(uint64_t h, uint32_t shift) {
    return (h * kGolden) >> shift;
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

// Eq. (2) in integer form, the feasibility mask and the cost C of Eq. (5)
// with Eqs. (3)-(4), for prefix length j on decode d.
struct PairCost {
    float cost;
    bool feas;
};

__device__ inline PairCost pair_cost(const Snap &s, uint32_t p, uint32_t d, uint32_t len, uint32_t j,
                                     float util, float load) {
    uint64_t s_eff = (uint64_t)s.bpt * (uint64_t)(len - s.block_tokens * j);
    uint64_t m = s.free_mem[d];
    bool feas = (m >= s.m_min) && (m - s.m_min >= s_eff);
    uint32_t tau = s.tier_map[(uint64_t)p * s.D + d] & 3u;
    float n = (float)s.n_inflight[tau * s.P + p];
    float t_x = ((float)s_eff * (1.0f + n)) / (s.bw[tau] * (1.0f - util)) + s.lat[tau];
    PairCost pc;
    pc.cost = t_x + load;
    pc.feas = feas;
    return pc;
}

__device__ inline uint64_t pack_key(float cost, uint32_t d) {
    return ((uint64_t)__float_as_uint(cost) << 32) | (uint64_t)d;
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

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl_xor(lo, m, kWave);
    hi = __shfl_xor(hi, m, kWave);
    return ((uint64_t)hi << 32) | lo;
}

__device__ inline uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) {
        uint64_t o = shfl_xor_u64(v, m);
        v = o < v ? o : v;
    }
    return v;
}

__device__ inline uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

__device__ inline uint64_t uniform_u64(uint64_t v) {
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Blocks are handed to the 8 XCDs round-robin; give each XCD a contiguous
// range of logical blocks so neighbouring requests share an L2.
__device__ inline uint32_t xcd_block(uint32_t b, uint32_t g) {
    const uint32_t nx = 8;
    uint32_t q = g / nx, rem = g % nx;
    uint32_t x = b % nx, i = b / nx;
    return x < rem ? x * (q + 1) + i : rem * (q + 1) + (x - rem) * q + i;
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

// First-miss prefix match of one request against 64 decodes (lanes), with
// W home-slot loads issued together per step.  `col` points at this lane's
// column of the slot-major table; the hash run is wave-uniform.
template <int W>
__device__ inline uint32_t prefix_match(const uint64_t *__restrict__ col, const Table &t,
                                        const uint64_t *lds_run, const uint64_t *__restrict__ g_run,
                                        uint32_t n, bool active) {
    uint32_t j = 0;
    bool alive = active;
    for (uint32_t i0 = 0; i0 < n; i0 += W) {
        if (!__any(alive)) break;
        uint64_t h[W], sl[W], key[W];
#pragma unroll
        for (int w = 0; w < W; ++w) {
            uint32_t i = i0 + w;
            uint64_t v = 0;
            if (i < n) v = i < (uint32_t)kStage ? lds_run[i] : g_run[i];
            h[w] = uniform_u64(v);
            sl[w] = home_slot(h[w], t.shift);
            key[w] = 0;
            if (alive && i < n) key[w] = col[sl[w] * t.pitch];
        }
#pragma unroll
        for (int w = 0; w < W; ++w) {
            if (i0 + w >= n) break;
            bool hit = alive && key[w] == h[w];
            bool pend = alive && key[w] != h[w] && key[w] != 0;
            uint64_t s2 = sl[w];
            while (__any(pend)) {
                s2 = (s2 + 1) & t.mask;
                if (pend) {
                    uint64_t k2 = col[s2 * t.pitch];
                    if (k2 == h[w]) {
                        hit = true;
                        pend = false;
                    } else if (k2 == 0) {
                        pend = false;
                    }
                }
            }
            alive = hit;
            j += alive ? 1u : 0u;
        }
    }
    return j;
}

// One wavefront per request; lanes are decodes c*64 + lane, c = 0..ceil(D/64)-1.
template <int K, int W, bool PAIRS>
__global__ __launch_bounds__(kBlock) void select_kernel(Snap s, Table t, Reqs rq, uint32_t k,
                                                        int32_t *__restrict__ out_idx,
                                                        float *__restrict__ out_score, PairOut po,
                                                        uint32_t *__restrict__ err) {
    __shared__ uint64_t run[kWavesPerBlock][kStage];
    const uint32_t wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);
    const uint32_t r = blk * kWavesPerBlock + wave;
    if (r >= rq.n_req) return;

    uint32_t p, len, n;
    uint64_t a;
    bool ok = request_ok(rq, s, r, p, len, a, n);
    bool zero = false;
    if (ok) {
        const uint64_t *g = rq.hashes + a;
        for (uint32_t i = lane; i < n; i += kWave) {
            uint64_t v = g[i];
            if (i < (uint32_t)kStage) run[wave][i] = v;
            zero |= (v == 0);
        }
    }
    const bool any_zero = __any(zero);
    if (!ok || any_zero) {
        if (lane < k) {
            out_idx[(uint64_t)r * k + lane] = -1;
            out_score[(uint64_t)r * k + lane] = __builtin_nanf("");
        }
        if (lane == 0) atomicOr(err, ok ? kErrZeroHash : kErrRequest);
        return;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    uint64_t best[K];
#pragma unroll
    for (int i = 0; i < K; ++i) best[i] = kEmptyKey;

    const uint64_t *g_run = rq.hashes + a;
    const uint32_t nchunk = (s.D + kWave - 1) / kWave;
    for (uint32_t c = 0; c < nchunk; ++c) {
        const uint32_t d = c * kWave + lane;
        const bool act = d < s.D;
        const uint32_t dd = act ? d : 0;
        uint32_t j = prefix_match<W>(t.keys + dd, t, run[wave], g_run, n, act);
        if (act) {
            float util = s.util[(uint64_t)p * s.D + d];
            PairCost pc = pair_cost(s, p, d, len, j, util, load_term(s, d));
            if (PAIRS) {
                uint64_t o = (uint64_t)r * s.D + d;
                if (po.j) po.j[o] = (uint16_t)j;
                if (po.feas) po.feas[o] = pc.feas ? 1 : 0;
                if (po.score) po.score[o] = pc.cost;
                if (po.jT) po.jT[(uint64_t)d * rq.n_req + r] = (uint16_t)j;
            }
            if (pc.feas) topk_insert<K>(best, pack_key(pc.cost, d));
        }
    }
    for (uint32_t i = 0; i < k; ++i) {
        uint64_t m = wave_min_u64(best[0]);
        if (best[0] == m && m != kEmptyKey) {
#pragma unroll
            for (int q = 0; q + 1 < K; ++q) best[q] = best[q + 1];
            best[K - 1] = kEmptyKey;
        }
        if (lane == 0) {
            out_idx[(uint64_t)r * k + i] = m == kEmptyKey ? -1 : (int32_t)(uint32_t)m;
            out_score[(uint64_t)r * k + i] = m == kEmptyKey ? __builtin_inff()
                                                            : __uint_as_float((uint32_t)(m >> 32));
        }
    }
}

// Ranking sweep: one thread per (request, scenario); decodes looped.
template <int K>
__global__ __launch_bounds__(256) void sweep_kernel(Snap s, Reqs rq, const float *__restrict__ util_scen,
                                                    const uint16_t *__restrict__ jT,
                                                    const int32_t *__restrict__ base_idx, uint32_t k,
                                                    int32_t *__restrict__ out_idx,
                                                    float *__restrict__ out_score,
                                                    unsigned long long *__restrict__ flips) {
    const uint32_t sc = blockIdx.y;
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    const bool act = r < rq.n_req;
    uint32_t tier_flip = 0, idx_flip = 0;
    if (act) {
        uint32_t p, len, n;
        uint64_t a;
        uint64_t o = ((uint64_t)sc * rq.n_req + r) * k;
        if (!request_ok(rq, s, r, p, len, a, n)) {
            for (uint32_t i = 0; i < k; ++i) {
                out_idx[o + i] = -1;
                out_score[o + i] = __builtin_nanf("");
            }
        } else {
            const float *u = util_scen + (uint64_t)sc * s.P * s.D + (uint64_t)p * s.D;
            uint64_t best[K];
#pragma unroll
            for (int i = 0; i < K; ++i) best[i] = kEmptyKey;
            for (uint32_t d = 0; d < s.D; ++d) {
                uint32_t j = jT[(uint64_t)d * rq.n_req + r];
                PairCost pc = pair_cost(s, p, d, len, j, u[d], load_term(s, d));
                if (pc.feas) topk_insert<K>(best, pack_key(pc.cost, d));
            }
            for (uint32_t i = 0; i < k; ++i) {
                uint64_t m = i < (uint32_t)K ? best[i] : kEmptyKey;
                out_idx[o + i] = m == kEmptyKey ? -1 : (int32_t)(uint32_t)m;
                out_score[o + i] = m == kEmptyKey ? __builtin_inff() : __uint_as_float((uint32_t)(m >> 32));
            }
            int32_t sel = best[0] == kEmptyKey ? -1 : (int32_t)(uint32_t)best[0];
            int32_t ref = base_idx[r];
            int ts = sel < 0 ? -1 : (int)s.tier_map[(uint64_t)p * s.D + (uint32_t)sel];
            int tr = ref < 0 ? -1 : (int)s.tier_map[(uint64_t)p * s.D + (uint32_t)ref];
            tier_flip = ts != tr;
            idx_flip = sel != ref;
        }
    }
    if (flips) {
        uint32_t a = wave_sum_u32(tier_flip), b = wave_sum_u32(idx_flip);
        if ((threadIdx.x % kWave) == 0) {
            if (a) atomicAdd(flips + 2 * sc, (unsigned long long)a);
            if (b) atomicAdd(flips + 2 * sc + 1, (unsigned long long)b);
        }
    }
}

// ------------------------------------------------------------------ table build

__global__ void count_zero_kernel(const uint64_t *__restrict__ h, uint64_t n, uint32_t *__restrict__ err) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    bool z = false;
    for (; i < n; i += stride) z |= h[i] == 0;
    if (__any(z) && (threadIdx.x % kWave) == 0) atomicOr(err, kErrZeroHash);
}

// Tiles of one decode's hash list: tile_dec[b], tile_beg[b], tile_end[b].
__global__ __launch_bounds__(256) void insert_kernel(uint64_t *__restrict__ keys, uint64_t mask, uint32_t shift,
                                                     uint32_t pitch, const uint64_t *__restrict__ h,
                                                     const uint32_t *__restrict__ tile_dec,
                                                     const uint64_t *__restrict__ tile_beg,
                                                     const uint64_t *__restrict__ tile_end,
                                                     uint32_t *__restrict__ err) {
    const uint32_t d = tile_dec[blockIdx.x];
    const uint64_t beg = tile_beg[blockIdx.x], end = tile_end[blockIdx.x];
    for (uint64_t i = beg + threadIdx.x; i < end; i += blockDim.x) {
        uint64_t key = h[i];
        uint64_t sl = home_slot(key, shift);
        bool done = false;
        for (uint64_t step = 0; step <= mask; ++step) {
            unsigned long long prev =
                atomicCAS((unsigned long long *)(keys + sl * pitch + d), 0ull, (unsigned long long)key);
            if (prev == 0ull || prev == key) {
                done = true;
                break;
            }
            sl = (sl + 1) & mask;
        }
        if (!done) atomicOr(err, kErrTableFull);
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

// Probe one (hash run, decode) pair by itself (one thread).
__device__ inline uint32_t prefix_match_one(const Table &t, uint32_t d, const uint64_t *__restrict__ run,
                                            uint32_t n) {
    uint32_t j = 0;
    for (; j < n; ++j) {
        uint64_t h = run[j];
        uint64_t sl = home_slot(h, t.shift);
        bool hit = false;
        for (uint64_t step = 0; step <= t.mask; ++step) {
            uint64_t key = t.keys[sl * t.pitch + d];
            if (key == h) {
                hit = true;
                break;
            }
            if (key == 0) break;
            sl = (sl + 1) & t.mask;
        }
        if (!hit || h == 0) break;
    }
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

}  // namespace

// ====================================================================== host side

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
    float bw[4] = {0, 0, 0, 0}, lat[4] = {0, 0, 0, 0};
    float t_a = 0, t_b = 0, alpha = 0;
    uint32_t beta_max = 0, bpt = 0, block_tokens = 1;
    uint64_t m_min = 0;
    // cache
    bool have_cache = false;
    uint32_t cache_D = 0;
    uint64_t *table = nullptr;
    uint64_t table_bytes = 0, cap = 0;
    uint32_t log2cap = 0, pitch = 0;
    // scratch
    uint32_t *errword = nullptr;          // request / selection errors (sticky)
    uint32_t *loadword = nullptr;         // validation flags of the load calls
    uint16_t *jT = nullptr;
    uint64_t jT_bytes = 0;
    int32_t *base_idx = nullptr;
    float *base_score = nullptr;
    uint64_t base_n = 0;
    uint32_t *cnt = nullptr, *adm = nullptr;
    unsigned long long *bytes = nullptr;
    uint32_t commit_P = 0, commit_D = 0;
    // timing
    bool timing = false;
    bool timed = false;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
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
    return s;
}

Table make_table(netkv_handle h) {
    Table t;
    t.keys = h->table;
    t.mask = h->cap - 1;
    t.shift = 64 - h->log2cap;
    t.pitch = h->pitch;
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

template <int K, int W>
void launch_select_k(const Snap &s, const Table &t, const Reqs &rq, uint32_t k, int32_t *idx,
                     float *score, const PairOut &po, bool pairs, uint32_t *err, hipStream_t st) {
    uint32_t grid = (rq.n_req + kWavesPerBlock - 1) / kWavesPerBlock;
    if (pairs)
        hipLaunchKernelGGL((select_kernel<K, W, true>), dim3(grid), dim3(kBlock), 0, st, s, t, rq, k, idx,
                           score, po, err);
    else
        hipLaunchKernelGGL((select_kernel<K, W, false>), dim3(grid), dim3(kBlock), 0, st, s, t, rq, k, idx,
                           score, po, err);
}

constexpr int kSpec = 4;   // home-slot loads issued together per probe step

void launch_select(const Snap &s, const Table &t, const Reqs &rq, uint32_t k, int32_t *idx, float *score,
                   const PairOut &po, bool pairs, uint32_t *err, hipStream_t st) {
    if (k <= 1) launch_select_k<1, kSpec>(s, t, rq, k, idx, score, po, pairs, err, st);
    else if (k <= 2) launch_select_k<2, kSpec>(s, t, rq, k, idx, score, po, pairs, err, st);
    else if (k <= 4) launch_select_k<4, kSpec>(s, t, rq, k, idx, score, po, pairs, err, st);
    else launch_select_k<8, kSpec>(s, t, rq, k, idx, score, po, pairs, err, st);
}

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

}  // namespace

// ------------------------------------------------------------------ API

extern "C" {

netkv_status netkv_create(netkv_handle *out, int device) {
    if (!out) return NETKV_EINVAL;
    *out = nullptr;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return NETKV_EINVAL;
    netkv_handle h = new netkv_ctx();
    h->device = device;
    DeviceGuard g(device);
    if (dalloc(h->errword, 1) != hipSuccess || dalloc(h->loadword, 1) != hipSuccess ||
        hipMemset(h->errword, 0, 4) != hipSuccess || hipMemset(h->loadword, 0, 4) != hipSuccess ||
        hipEventCreate(&h->ev0) != hipSuccess || hipEventCreate(&h->ev1) != hipSuccess) {
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
        dfree(h->tier_map);
        dfree(h->util);
        dfree(h->n_inflight);
        dfree(h->free_mem);
        dfree(h->queue);
        dfree(h->batch);
        dfree(h->adm_prev);
        dfree(h->table);
        dfree(h->errword);
        dfree(h->loadword);
        dfree(h->jT);
        dfree(h->base_idx);
        dfree(h->base_score);
        dfree(h->cnt);
        dfree(h->adm);
        dfree(h->bytes);
        if (h->ev0) (void)hipEventDestroy(h->ev0);
        if (h->ev1) (void)hipEventDestroy(h->ev1);
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
    if ((uint64_t)P * D > (1ull << 34)) return fail(h, NETKV_EINVAL, "P*D too large");
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
    dfree(h->tier_map); dfree(h->util); dfree(h->n_inflight); dfree(h->free_mem);
    dfree(h->adm_prev); dfree(h->queue); dfree(h->batch);
    h->tier_map = tm; h->util = ut; h->n_inflight = ni; h->free_mem = fm;
    h->adm_prev = ap; h->queue = qd; h->batch = bs;
    h->P = P;
    h->D = D;
    for (int i = 0; i < 4; ++i) {
        h->bw[i] = (float)o->tier_bw[i];
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
    uint64_t maxn = 0;
    for (uint32_t d = 0; d < n_decode; ++d) {
        if (off[d + 1] < off[d]) return fail(h, NETKV_EINVAL, "hash_off decreases at decode %u", d);
        maxn = std::max(maxn, off[d + 1] - off[d]);
    }
    if (off[n_decode] > n_hashes) return fail(h, NETKV_EINVAL, "hash_off[n_decode] exceeds n_hashes");
    uint64_t need = (uint64_t)std::ceil((double)maxn / (double)max_load_factor);
    uint32_t log2cap = 4;
    while ((1ull << log2cap) < need || (1ull << log2cap) <= maxn) {
        ++log2cap;
        if (log2cap > 31) return fail(h, NETKV_ECAPACITY, "a table would need more than 2^31 slots");
    }
    const uint64_t cap = 1ull << log2cap;
    const uint32_t pitch = (n_decode + 15u) & ~15u;
    const uint64_t tbytes = cap * pitch * 8ull;
    // tiles of at most 4096 hashes, each within one decode
    const uint64_t kTile = 4096;
    std::vector<uint32_t> tdec;
    std::vector<uint64_t> tbeg, tend;
    for (uint32_t d = 0; d < n_decode; ++d)
        for (uint64_t b = off[d]; b < off[d + 1]; b += kTile) {
            tdec.push_back(d);
            tbeg.push_back(b);
            tend.push_back(std::min(off[d + 1], b + kTile));
        }
    const uint64_t first = off[0], total = off[n_decode] - off[0];
    uint64_t *dh = nullptr, *dbeg = nullptr, *dend = nullptr, *tab = nullptr;
    uint32_t *ddec = nullptr;
    auto cleanup = [&]() { dfree(dh); dfree(dbeg); dfree(dend); dfree(ddec); dfree(tab); };
    // the device copy keeps the caller's absolute offsets valid: copy from `first`
    if (dalloc(dh, off[n_decode]) != hipSuccess || dalloc(dbeg, tbeg.size()) != hipSuccess ||
        dalloc(dend, tend.size()) != hipSuccess || dalloc(ddec, tdec.size()) != hipSuccess) {
        cleanup();
        return fail(h, NETKV_ENOMEM, "staging allocation failed");
    }
    hipError_t e = hipSuccess;
    if (total) e = hipMemcpyAsync(dh + first, hashes + first, 8ull * total, hipMemcpyDefault, st);
    if (e == hipSuccess && !tdec.empty()) e = hipMemcpyAsync(ddec, tdec.data(), 4ull * tdec.size(), hipMemcpyHostToDevice, st);
    if (e == hipSuccess && !tbeg.empty()) e = hipMemcpyAsync(dbeg, tbeg.data(), 8ull * tbeg.size(), hipMemcpyHostToDevice, st);
    if (e == hipSuccess && !tend.empty()) e = hipMemcpyAsync(dend, tend.data(), 8ull * tend.size(), hipMemcpyHostToDevice, st);
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
    // release the old table first: the new one may be large
    dfree(h->table);
    h->have_cache = false;
    e = dalloc(tab, cap * pitch);
    if (e != hipSuccess) {
        cleanup();
        return fail(h, NETKV_ENOMEM, "table allocation of %llu bytes failed", (unsigned long long)tbytes);
    }
    e = hipMemsetAsync(tab, 0, tbytes, st);
    if (e == hipSuccess && !tdec.empty()) {
        hipLaunchKernelGGL(insert_kernel, dim3((uint32_t)tdec.size()), dim3(256), 0, st, tab, cap - 1,
                           64u - log2cap, pitch, (const uint64_t *)dh, (const uint32_t *)ddec,
                           (const uint64_t *)dbeg, (const uint64_t *)dend, h->loadword);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, h->loadword, 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    dfree(dh); dfree(dbeg); dfree(dend); dfree(ddec);
    if (e != hipSuccess || bad) {
        dfree(tab);
        return e != hipSuccess ? fail(h, NETKV_EDEVICE, "table build failed: %s", hipGetErrorString(e))
                               : fail(h, NETKV_ECAPACITY, "table build ran out of slots");
    }
    h->table = tab;
    h->cap = cap;
    h->log2cap = log2cap;
    h->pitch = pitch;
    h->table_bytes = tbytes;
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
    PairOut po{nullptr, nullptr, nullptr, nullptr};
    bool want_pairs = false;
    if (pairs) {
        po.j = pairs->prefix_blocks;
        po.feas = pairs->feasible;
        po.score = pairs->score;
        want_pairs = po.j || po.feas || po.score;
    }
    if (h->timing) HIPCHK(h, hipEventRecord(h->ev0, s));
    launch_select(make_snap(h), make_table(h), make_reqs(req), k, out_idx, out_score, po, want_pairs, h->errword, s);
    HIPCHK(h, hipGetLastError());
    if (h->timing) {
        HIPCHK(h, hipEventRecord(h->ev1, s));
        h->timed = true;
    }
    return NETKV_OK;
}

netkv_status netkv_rank_sweep(netkv_handle h, const netkv_requests_t *req, uint32_t n_scen, const float *util_scen,
                              uint32_t k, int32_t *out_idx, float *out_score, uint64_t *out_flips, void *stream) {
    if (!h) return NETKV_EINVAL;
    h->err.clear();
    netkv_status st = check_requests(h, req);
    if (st) return st;
    if (k < 1 || k > 8) return fail(h, NETKV_EINVAL, "k must be in [1, 8]");
    if (n_scen > 65535) return fail(h, NETKV_EINVAL, "n_scen must be <= 65535");
    if (n_scen && req->n_req && (!util_scen || !out_idx || !out_score))
        return fail(h, NETKV_EINVAL, "util_scen, out_idx and out_score must not be NULL");
    if ((st = ready(h))) return st;
    if (req->n_req == 0 || n_scen == 0) return NETKV_OK;
    DeviceGuard g(h->device);
    hipStream_t s = (hipStream_t)stream;
    const uint64_t R = req->n_req, D = h->D;
    if (h->jT_bytes < R * D * 2) {
        dfree(h->jT);
        h->jT_bytes = 0;
        HIPCHK(h, dalloc(h->jT, R * D));
        h->jT_bytes = R * D * 2;
    }
    if (h->base_n < R) {
        dfree(h->base_idx);
        dfree(h->base_score);
        h->base_n = 0;
        HIPCHK(h, dalloc(h->base_idx, R));
        HIPCHK(h, dalloc(h->base_score, R));
        h->base_n = R;
    }
    Snap sn = make_snap(h);
    Reqs rq = make_reqs(req);
    // prefix lengths (transposed) and the selection under the loaded congestion
    PairOut po{nullptr, nullptr, nullptr, h->jT};
    launch_select(sn, make_table(h), rq, 1, h->base_idx, h->base_score, po, true, h->errword, s);
    HIPCHK(h, hipGetLastError());
    if (out_flips) {
        hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(2ull * n_scen, 256)), dim3(256), 0, s, out_flips,
                           2ull * n_scen, 0ull);
        HIPCHK(h, hipGetLastError());
    }
    if (h->timing) HIPCHK(h, hipEventRecord(h->ev0, s));
    dim3 grid((uint32_t)((R + 255) / 256), n_scen);
    unsigned long long *fl = (unsigned long long *)out_flips;
    if (k <= 1)
        hipLaunchKernelGGL(sweep_kernel<1>, grid, dim3(256), 0, s, sn, rq, util_scen, h->jT, h->base_idx, k, out_idx,
                           out_score, fl);
    else if (k <= 2)
        hipLaunchKernelGGL(sweep_kernel<2>, grid, dim3(256), 0, s, sn, rq, util_scen, h->jT, h->base_idx, k, out_idx,
                           out_score, fl);
    else if (k <= 4)
        hipLaunchKernelGGL(sweep_kernel<4>, grid, dim3(256), 0, s, sn, rq, util_scen, h->jT, h->base_idx, k, out_idx,
                           out_score, fl);
    else
        hipLaunchKernelGGL(sweep_kernel<8>, grid, dim3(256), 0, s, sn, rq, util_scen, h->jT, h->base_idx, k, out_idx,
                           out_score, fl);
    HIPCHK(h, hipGetLastError());
    if (h->timing) {
        HIPCHK(h, hipEventRecord(h->ev1, s));
        h->timed = true;
    }
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
        return fail(h, NETKV_EINVAL, "input errors:%s%s%s%s", (e & kErrRequest) ? " inconsistent request header" : "",
                    (e & kErrZeroHash) ? " request hash 0" : "", (e & kErrSelection) ? " selection index >= D" : "",
                    (e & kErrTableFull) ? " table full" : "");
    return NETKV_OK;
}

netkv_status netkv_set_timing(netkv_handle h, int enable) {
    if (!h) return NETKV_EINVAL;
    h->timing = enable != 0;
    h->timed = false;
    return NETKV_OK;
}

netkv_status netkv_kernel_ms(netkv_handle h, float *ms) {
    if (!h || !ms) return NETKV_EINVAL;
    h->err.clear();
    if (!h->timed) return fail(h, NETKV_ENOTREADY, "no timed kernel yet");
    DeviceGuard g(h->device);
    HIPCHK(h, hipEventSynchronize(h->ev1));
    HIPCHK(h, hipEventElapsedTime(ms, h->ev0, h->ev1));
    return NETKV_OK;
}

netkv_status netkv_cache_info(netkv_handle h, uint64_t *slots_per_decode, uint64_t *table_bytes) {
    if (!h) return NETKV_EINVAL;
    if (!h->have_cache) return fail(h, NETKV_ENOTREADY, "no cache loaded");
    if (slots_per_decode) *slots_per_decode = h->cap;
    if (table_bytes) *table_bytes = h->table_bytes;
    return NETKV_OK;
}

}  // extern "C"

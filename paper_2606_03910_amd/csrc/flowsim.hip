// Flow-level transfer simulation (Sec. VI-B, the evaluation simulator's
// network model) for MI355X (gfx950).
//
// KV transfers are flows over the links of their paths.  Each link is
// shared max-min fairly among the flows crossing it, and every flow arrival
// or completion re-evaluates the allocation of all flows in progress;
// background traffic is a steady utilisation already taken out of each
// link's capacity (the section's mean-field model).  The allocation is the
// max-min fair one, computed by progressive filling: all unfrozen flows'
// rates rise together by the largest amount every link still allows; the
// flows crossing a link that this fills stop there; repeat.
//
// One workgroup runs one instance (a flow set on its links) through all its
// events; the instances of a call are independent (other congestion draws,
// other batches).  Inside a workgroup, threads take links and flows in
// strides, and workgroup reductions give the minimum raise, the next event
// and the counts.  Before the simulation each instance's flows are sorted
// by arrival time (rocPRIM's segmented radix sort, which only orders work),
// so that a pass takes its arrivals from the head of that order and keeps
// the list of flows in progress from pass to pass: its cost follows the
// flows in progress, not the instance's size.  Every quantity is fp64 and every operation is written
// out in order with contraction off, so the results equal those of a
// sequential implementation of the same steps bit for bit (minima do not
// depend on the reduction order; link counts are integers).

#include <hip/hip_runtime.h>
#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_segmented_radix_sort.hpp>

#include <cmath>
#include <cstdint>

#include "netkv.h"
#include "netkv_internal.h"

namespace {

constexpr int kSimThreads = 256;
constexpr int kWave = 64;
constexpr int kSimWaves = kSimThreads / kWave;
constexpr uint32_t kSimLdsLinks = 2048;   // instances with at most this many links keep them in LDS
constexpr uint32_t kPathRegs = 6;         // path links a wavefront-path lane keeps in registers
constexpr uint32_t kLinkRegs = 2;         // links per thread whose round state the workgroup path keeps in registers
constexpr uint32_t kWaveLinkRegs = 5;     // the same per lane of the wavefront run

// flow states
constexpr uint8_t kWaiting = 0, kMoving = 1, kDone = 2;
// freeze marks of a moving flow within one allocation
constexpr uint8_t kFree = 0, kFrozen = 1, kJustFrozen = 2;

struct SimArgs {
    uint32_t n_links;
    const double *cap;          // [n_inst][n_links]
    const uint64_t *flow_off;   // [n_inst + 1]
    uint64_t n_flows;
    const uint64_t *path_off;   // [n_flows + 1]
    const uint32_t *path;
    uint64_t n_path;
    const double *bytes, *start;
    double *finish;
    uint64_t *stats;   // [n_inst][3]: allocations, filling rounds, moving flows summed over allocations
    // work: per flow, and per link of every instance (when not in LDS)
    double *remaining, *rate;
    uint8_t *state, *frz;
    uint32_t *mlist, *mlist2;   // [n_flows] the moving flows of each instance (its own range), in turn
    const uint32_t *arr;        // [n_flows] each instance's flows (offsets) in order of arrival
    const uint64_t *skey;       // [n_flows] their arrival times as sort keys, in that order
    const uint32_t *bad_off;    // nonzero: flow_off is not a valid partition of the flows
    const uint32_t *order;      // [n_inst] the instance of each workgroup, heaviest first (or null)
    double *g_rem;
    uint32_t *g_cnt, *g_lk;
    uint8_t *g_sat;
    uint32_t *err;
};

__device__ inline double dmin(double a, double b) { return b < a ? b : a; }

// Wavefront reductions by DPP (every lane active): pairs and pairs of
// pairs within each quad, rotations by 4 and 8 within each row of 16, then
// the last lane of row 0 into row 1 and of row 2 into row 3, and of row 1
// into rows 2 and 3; lane 63 then holds the result, which is read back to
// every lane.  A lane without a source takes the operation's identity.
// (DPP controls: quad_perm 0xB1 and 0x4E, row_ror 0x124 and 0x128,
// row_bcast 0x142 and 0x143.)
template <int CTRL, int ROWS>
__device__ inline double dpp_f64(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROWS, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0x7FF00000, (int)(uint32_t)(b >> 32), CTRL, ROWS, 0xF,
                                                              false);   // +infinity where there is no source
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ inline double wave_min_f64(double v) {
    v = dmin(v, dpp_f64<0xB1, 0xF>(v));
    v = dmin(v, dpp_f64<0x4E, 0xF>(v));
    v = dmin(v, dpp_f64<0x124, 0xF>(v));
    v = dmin(v, dpp_f64<0x128, 0xF>(v));
    v = dmin(v, dpp_f64<0x142, 0xA>(v));
    v = dmin(v, dpp_f64<0x143, 0xC>(v));
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 63);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ inline uint32_t wave_sum_u32(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Ordering of one wavefront's LDS and memory accesses between the phases
// of a filling round (lanes read what other lanes of the wavefront wrote).
__device__ inline void wave_phase() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup"); }

// The arrival time of a key of the arrival sort (the inverse of its map).
__device__ inline double key_time(uint64_t k) {
    return __longlong_as_double((long long)((k >> 63) ? (k ^ (1ull << 63)) : ~k));
}

using lmask = uint64_t;
__device__ inline lmask ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
// set bits of m below this lane
__device__ inline uint32_t below(lmask m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
// lane i's v goes to lane dst (a permutation of the lanes)
__device__ inline uint32_t send_u32(uint32_t v, uint32_t dst) {
    return (uint32_t)__builtin_amdgcn_ds_permute((int)(dst * 4u), (int)v);
}
__device__ inline uint64_t send_u64(uint64_t v, uint32_t dst) {
    return ((uint64_t)send_u32((uint32_t)(v >> 32), dst) << 32) | send_u32((uint32_t)v, dst);
}

// Where an instance stands when the wavefront run and the workgroup passes
// hand over to each other (in LDS; the moving flows are then in the device
// list `list`).
struct SimCtl {
    double t, nx;          // the clock; the next arrival (infinity: none left)
    uint64_t ap;           // arrivals taken (a prefix of the arrival order)
    uint64_t left;         // flows not completed
    uint64_t pass;         // passes so far (bounded)
    uint64_t events, rounds, moving;
    uint32_t na;           // moving flows
    uint32_t list;         // the device list that holds them: 0 mlist, 1 mlist2
    uint32_t mode;         // kRunWave, kRunGroup or kRunEnd
    uint32_t resume;       // the current pass has taken its arrivals already
    uint32_t stall;        // an iteration bound was reached
};
constexpr uint32_t kRunWave = 0, kRunGroup = 1, kRunEnd = 2;

// The instance's passes while at most one wavefront of flows moves, run by
// wavefront 0 alone.  Lane i keeps moving flow i (its offset, path and
// remaining size) in registers from pass to pass.  A pass takes the
// arrivals that are due into free lanes (from the sorted arrival order),
// counts the flows on their links, runs the filling rounds and the event,
// and moves the flows that are still in progress to the lowest lanes.  When
// more flows are due than lanes are free, the lanes' flows go to the device
// list and the workgroup passes take over.  Each flow and each link goes
// through the operations of the workgroup pass, in the same order.
__device__ void wave_run(const SimArgs &a, uint64_t f0, uint64_t nf, const uint32_t *arr, const uint64_t *skey,
                         double *rem, uint32_t *cnt, uint8_t *sat, uint32_t *lk, const double *lcap,
                         uint32_t *n_lk, SimCtl &c, uint32_t lane) {
#pragma clang fp contract(off)
    double t = c.t, nx = c.nx;
    uint64_t ap = c.ap, left = c.left, pass = c.pass, events = c.events, rounds = c.rounds, moving = c.moving;
    uint32_t na = c.na;
    bool resume = c.resume != 0;
    uint32_t *list = (c.list ? a.mlist2 : a.mlist) + f0;
    uint32_t o = 0, plen = 0;
    uint64_t p0 = 0;
    uint32_t pl[kPathRegs];
    double rm = 0.0;
    auto take = [&](uint32_t off) {   // the flow's path (its first kPathRegs links in registers)
        const uint64_t f = f0 + off;
        p0 = a.path_off[f];
        plen = (uint32_t)(a.path_off[f + 1] - p0);
#pragma unroll
        for (uint32_t u = 0; u < kPathRegs; ++u) pl[u] = u < plen ? a.path[p0 + u] : 0u;
    };
    auto link = [&](uint32_t u) { return u < kPathRegs ? pl[u] : a.path[p0 + u]; };
#pragma unroll
    for (uint32_t u = 0; u < kPathRegs; ++u) pl[u] = 0u;
    bool has = lane < na;
    if (has) {
        o = list[lane];
        take(o);
        rm = a.remaining[f0 + o];
    }
    uint32_t mode = kRunEnd, stall = 0;
    for (;; ++pass) {
        if (left == 0) break;
        if (!resume) {
            if (pass > 2 * nf + 4) {
                stall = 1;
                break;
            }
            if (t >= nx) {
                // the arrivals that are due: lane na + j takes arrival ap + j
                const uint64_t q = ap + (uint64_t)(lane - na);
                const bool cand = lane >= na && q < nf;
                double sq = INFINITY;
                uint32_t oq = 0;
                if (cand) {
                    sq = key_time(skey[f0 + q]);
                    oq = arr[q];
                }
                const bool in = cand && sq <= t;   // a prefix of the free lanes (the order is sorted)
                const uint32_t cn = (uint32_t)__builtin_popcountll(ballot(in));
                double nx2;
                if (na + cn < (uint32_t)kWave) nx2 = __shfl(sq, (int)(na + cn), kWave);
                else nx2 = ap + cn < nf ? key_time(skey[f0 + ap + cn]) : INFINITY;
                if (na + cn == (uint32_t)kWave && nx2 <= t) {
                    mode = kRunGroup;   // more flows due than lanes: the workgroup takes this pass
                    break;
                }
                if (in) {
                    o = oq;
                    take(o);
                    rm = a.bytes[f0 + o];
                    a.state[f0 + o] = kMoving;
                }
                ap += cn;
                na += cn;
                has = lane < na;
                nx = nx2;
            }
        }
        resume = false;
        if (na == 0) {
            t = nx;
            continue;
        }
        // the flows on their links (a link's first count lists it and resets its capacity)
        if (has) {
            for (uint32_t u = 0; u < plen; ++u) {
                const uint32_t l = link(u);
                if (atomicAdd(&cnt[l], 1u) == 0) {
                    rem[l] = lcap[l];
                    lk[atomicAdd(n_lk, 1u)] = l;
                }
            }
        }
        wave_phase();
        const uint32_t nl = *n_lk;
        // progressive filling
        bool frozen = !has;
        double level = 0.0, rt = 0.0;
        uint32_t rd = 0;
        for (;;) {
            if (!__any(!frozen)) break;
            if (rd > na) {   // every round freezes at least one flow
                stall = 1;
                break;
            }
            // the largest equal raise every link still allows; the lane's
            // first kWaveLinkRegs links keep their id, count, capacity left
            // and share for the update
            double sh = INFINITY;
            uint32_t ll[kWaveLinkRegs], lc[kWaveLinkRegs];
            double lr[kWaveLinkRegs], ls[kWaveLinkRegs];
#pragma unroll
            for (uint32_t k = 0; k < kWaveLinkRegs; ++k) {
                const uint32_t i = lane + k * kWave;
                ll[k] = 0;
                lc[k] = 0;
                lr[k] = 0.0;
                ls[k] = INFINITY;
                if (i < nl) {
                    ll[k] = lk[i];
                    lc[k] = cnt[ll[k]];
                    if (lc[k] > 0) {
                        lr[k] = rem[ll[k]];
                        ls[k] = lr[k] / (double)lc[k];
                        sh = dmin(sh, ls[k]);
                    }
                }
            }
            for (uint32_t i = lane + kWaveLinkRegs * kWave; i < nl; i += kWave) {
                const uint32_t l = lk[i];
                const uint32_t k = cnt[l];
                if (k > 0) sh = dmin(sh, rem[l] / (double)k);
            }
            const double inc = wave_min_f64(sh);
            // links that the raise fills, and the capacity left on each
#pragma unroll
            for (uint32_t k = 0; k < kWaveLinkRegs; ++k) {
                if (lane + k * kWave < nl) {
                    uint8_t full = 0;
                    if (lc[k] > 0) {
                        full = ls[k] == inc ? 1 : 0;
                        const double used = inc * (double)lc[k];
                        const double lf = lr[k] - used;
                        rem[ll[k]] = lf > 0.0 ? lf : 0.0;
                    }
                    sat[ll[k]] = full;
                }
            }
            for (uint32_t i = lane + kWaveLinkRegs * kWave; i < nl; i += kWave) {
                const uint32_t l = lk[i];
                const uint32_t k = cnt[l];
                uint8_t full = 0;
                if (k > 0) {
                    const double r = rem[l];
                    full = r / (double)k == inc ? 1 : 0;
                    const double used = inc * (double)k;
                    const double lf = r - used;
                    rem[l] = lf > 0.0 ? lf : 0.0;
                }
                sat[l] = full;
            }
            level = level + inc;
            wave_phase();
            // flows crossing a filled link stop at the current level
            bool just = false;
            if (!frozen) {
                uint8_t hit = 0;
                for (uint32_t u = 0; u < plen; ++u) hit |= sat[link(u)];
                if (hit) {
                    just = true;
                    frozen = true;
                    rt = level;
                }
            }
            wave_phase();
            if (just)
                for (uint32_t u = 0; u < plen; ++u) atomicSub(&cnt[link(u)], 1u);
            wave_phase();
            ++rd;
        }
        rounds += rd;
        if (stall) break;
        // the next event: the earliest completion, or the next arrival
        bool done = false;
        const double dtc = wave_min_f64(has ? rm / rt : INFINITY);
        if (dtc <= nx - t) {
            if (has) {
                if (rm / rt == dtc) {
                    a.state[f0 + o] = kDone;
                    a.finish[f0 + o] = t + dtc;
                    done = true;
                } else {
                    const double moved = rt * dtc;
                    const double r = rm - moved;
                    rm = r > 0.0 ? r : 0.0;
                }
            }
            t = t + dtc;
        } else {
            const double dt = nx - t;
            if (has) {
                const double moved = rt * dt;
                const double r = rm - moved;
                rm = r > 0.0 ? r : 0.0;
            }
            t = nx;
        }
        ++events;
        moving += na;
        if (lane == 0) *n_lk = 0;   // every lane has read the link count
        wave_phase();
        const lmask gone = ballot(done);
        if (gone) {
            // the flows still in progress to the lowest lanes, the others after them
            const lmask keep = ballot(has && !done);
            const uint32_t ns = (uint32_t)__builtin_popcountll(keep);
            const uint32_t dst = (has && !done) ? below(keep) : ns + below(~keep);
            o = send_u32(o, dst);
            plen = send_u32(plen, dst);
            p0 = send_u64(p0, dst);
#pragma unroll
            for (uint32_t u = 0; u < kPathRegs; ++u) pl[u] = send_u32(pl[u], dst);
            rm = __longlong_as_double((long long)send_u64((uint64_t)__double_as_longlong(rm), dst));
            left -= (uint64_t)__builtin_popcountll(gone);
            na = ns;
            has = lane < na;
        }
    }
    if (mode == kRunGroup && has) {
        list[lane] = o;
        a.remaining[f0 + o] = rm;
    }
    if (lane == 0) {
        c.t = t;
        c.nx = nx;
        c.ap = ap;
        c.left = left;
        c.pass = pass;
        c.events = events;
        c.rounds = rounds;
        c.moving = moving;
        c.na = na;
        c.mode = stall ? kRunEnd : mode;
        c.resume = 0;
        c.stall = stall;
    }
}

// Bytes of the link state an instance keeps in LDS: per link the capacity
// left and the capacity (fp64), the flow count and the list entry (u32),
// and the filled mark (u8).
__host__ __device__ inline uint32_t lds_link_bytes(uint32_t L) { return L * (8u + 8u + 4u + 4u + 1u); }

template <bool LDS>
__global__ __launch_bounds__(kSimThreads) void flow_sim_kernel(SimArgs a) {
#pragma clang fp contract(off)
    __shared__ double red_d[2][kSimWaves];
    __shared__ uint32_t red_u[2][kSimWaves];
    __shared__ uint32_t n_mv, n_lk;
    __shared__ SimCtl ctl;
    extern __shared__ __align__(8) unsigned char dyn[];   // the link state in LDS mode
    const uint32_t tid = threadIdx.x, lane = tid % 64, w = tid / 64;
    const uint32_t inst = a.order ? a.order[blockIdx.x] : blockIdx.x;
    const uint32_t L = a.n_links;
    const uint64_t f0 = a.flow_off[inst], f1 = a.flow_off[inst + 1];
    const double *cap = a.cap + (uint64_t)inst * L;
    double *rem = LDS ? (double *)dyn : a.g_rem + (uint64_t)inst * L;
    double *lcap = LDS ? (double *)dyn + L : nullptr;
    uint32_t *cnt = LDS ? (uint32_t *)(dyn + 16u * L) : a.g_cnt + (uint64_t)inst * L;
    uint32_t *lk = LDS ? (uint32_t *)(dyn + 20u * L) : a.g_lk + (uint64_t)inst * L;
    uint8_t *sat = LDS ? dyn + 24u * L : a.g_sat + (uint64_t)inst * L;
    // workgroup reductions: one barrier each; two buffers used in turn, so a
    // buffer is written again only after the next reduction's barrier,
    // which every thread reaches after reading it
    uint32_t par = 0;
    auto bmin = [&](double v) {
        v = wave_min_f64(v);
        if (lane == 0) red_d[par][w] = v;
        __syncthreads();
        double m = red_d[par][0];
#pragma unroll
        for (int q = 1; q < kSimWaves; ++q) m = dmin(m, red_d[par][q]);
        par ^= 1u;
        return m;
    };
    auto bsum = [&](uint32_t v) {
        v = wave_sum_u32(v);
        if (lane == 0) red_u[par][w] = v;
        __syncthreads();
        uint32_t m = red_u[par][0];
#pragma unroll
        for (int q = 1; q < kSimWaves; ++q) m += red_u[par][q];
        par ^= 1u;
        return m;
    };
    // the instance's input, checked before any simulation (offsets that are
    // not a partition of the flows invalidate every instance of the call)
    const bool range_ok = f0 <= f1 && f1 <= a.n_flows;
    uint32_t bad = range_ok && *a.bad_off == 0 ? 0u : 1u;
    for (uint32_t l = tid; l < L; l += kSimThreads) {
        const double c = cap[l];
        if (!(c > 0.0) || !isfinite(c)) bad = 1;
    }
    for (uint64_t f = f0 + tid; range_ok && f < f1; f += kSimThreads) {
        const uint64_t p0 = a.path_off[f], p1 = a.path_off[f + 1];
        if (!(p1 > p0) || p1 > a.n_path) {
            bad = 1;
        } else {
            for (uint64_t q = p0; q < p1; ++q)
                if (a.path[q] >= L) bad = 1;
        }
        const double b = a.bytes[f], s = a.start[f];
        if (!(b >= 0.0) || !isfinite(b) || !isfinite(s)) bad = 1;
    }
    if (bsum(bad)) {
        for (uint64_t f = f0 + tid; range_ok && f < f1; f += kSimThreads) a.finish[f] = NAN;
        if (tid == 0) {
            atomicOr(a.err, kErrFlowBit);
            if (a.stats)
                for (int q = 0; q < 3; ++q) a.stats[3ull * inst + q] = 0;
        }
        return;
    }
    // flows wait for their arrival; the clock starts at the first one.
    // Link counts start at 0 and return to 0 at the end of every allocation
    // (every flow counted on a link is frozen and uncounted again).
    for (uint32_t l = tid; l < L; l += kSimThreads) {
        cnt[l] = 0;
        if (LDS) lcap[l] = cap[l];
    }
    for (uint64_t f = f0 + tid; f < f1; f += kSimThreads) {
        a.state[f] = kWaiting;
        a.frz[f] = kFree;
        a.remaining[f] = a.bytes[f];
    }
    const uint64_t nf = f1 - f0;   // < 2^32 (the call's flows are)
    const uint32_t *arr = a.arr + f0;
    if (tid == 0) {
        n_lk = 0;
        ctl.t = nf ? key_time(a.skey[f0]) : INFINITY;   // the first arrival
        ctl.nx = ctl.t;
        ctl.ap = 0;
        ctl.left = nf;
        ctl.pass = 0;
        ctl.events = ctl.rounds = ctl.moving = 0;
        ctl.na = 0;
        ctl.list = 0;
        ctl.mode = nf ? kRunWave : kRunEnd;
        ctl.resume = 0;
        ctl.stall = 0;
    }
    __syncthreads();
    // the wavefront run while few flows move, the workgroup passes while
    // more do, handing over through ctl (each side reads it after the
    // barrier that follows the other side's writes)
    for (;;) {
        const uint32_t mode = ctl.mode;
        __syncthreads();   // every thread has read the mode before it changes
        if (mode == kRunEnd) break;
        if (mode == kRunWave) {
            if (w == 0)
                wave_run(a, f0, nf, arr, a.skey, rem, cnt, sat, lk, LDS ? (const double *)lcap : cap, &n_lk, ctl,
                         lane);
            __syncthreads();
            continue;
        }
        // workgroup passes: the moving flows in the device list mv (pass
        // state in every thread's registers, the same in all of them)
        double t = ctl.t;
        uint64_t ap = ctl.ap, left = ctl.left, pass = ctl.pass;
        uint64_t events = ctl.events, rounds = ctl.rounds, moving = ctl.moving;
        uint32_t na = ctl.na, cur = ctl.list;
        uint32_t *mv = (cur ? a.mlist2 : a.mlist) + f0, *mv2 = (cur ? a.mlist : a.mlist2) + f0;
        uint32_t next = kRunEnd, stall = 0;
        double nx = INFINITY;
        for (;; ++pass) {
            if (left == 0) break;
            if (pass > 2 * nf + 4) {
                stall = 1;
                break;
            }
            if (tid == 0) {
                n_mv = 0;
                n_lk = 0;
            }
            __syncthreads();   // the list counters' previous uses all precede the last barrier
            // this pass's moving flows: the previous list without the flows
            // that completed, then the flows that have arrived by t (a prefix
            // of the rest of the arrival order); the next arrival
            for (uint32_t i = tid; i < na; i += kSimThreads) {
                const uint32_t o = mv[i];
                if (a.state[f0 + o] != kDone) mv2[atomicAdd(&n_mv, 1u)] = o;
            }
            for (;;) {
                const uint64_t q = ap + tid;
                uint32_t in = 0;
                if (q < nf) {
                    const uint32_t o = arr[q];
                    if (a.start[f0 + o] <= t) {
                        a.state[f0 + o] = kMoving;
                        mv2[atomicAdd(&n_mv, 1u)] = o;
                        in = 1;
                    }
                }
                const uint32_t c = bsum(in);   // its barrier also orders the list writes before n_mv is read
                ap += c;
                if (c < (uint32_t)kSimThreads) break;
            }
            nx = ap < nf ? a.start[f0 + arr[ap]] : INFINITY;
            na = n_mv;
            {
                uint32_t *x = mv;
                mv = mv2;
                mv2 = x;
                cur ^= 1u;
            }
            if (na <= (uint32_t)kWave) {
                // few enough for the wavefront run, which finishes this pass
                next = kRunWave;
                break;
            }
            if (na <= (uint32_t)kSimThreads) {
                // at most one flow per thread: the thread keeps its flow's
                // path, freeze mark, rate and remaining size in registers
                // for the pass (the operations of the general case below)
                const bool has = tid < na;
                uint64_t f = 0, p0 = 0;
                uint32_t plen = 0;
                uint32_t pl[kPathRegs];
#pragma unroll
                for (uint32_t u = 0; u < kPathRegs; ++u) pl[u] = 0u;
                double rm = 0.0, rt = 0.0;
                if (has) {
                    f = f0 + mv[tid];
                    p0 = a.path_off[f];
                    plen = (uint32_t)(a.path_off[f + 1] - p0);
#pragma unroll
                    for (uint32_t u = 0; u < kPathRegs; ++u) pl[u] = u < plen ? a.path[p0 + u] : 0u;
                    rm = a.remaining[f];
                }
                auto link = [&](uint32_t u) { return u < kPathRegs ? pl[u] : a.path[p0 + u]; };
                if (has) {
                    for (uint32_t u = 0; u < plen; ++u) {
                        const uint32_t l = link(u);
                        if (atomicAdd(&cnt[l], 1u) == 0) {
                            rem[l] = LDS ? lcap[l] : cap[l];
                            lk[atomicAdd(&n_lk, 1u)] = l;
                        }
                    }
                }
                __syncthreads();
                const uint32_t nl = n_lk;
                bool frozen = !has;
                double level = 0.0;
                // every flow crosses a link, so the least share below is
                // infinite exactly when every flow is frozen
                for (uint32_t round = 0;; ++round) {
                    // the largest equal raise every link still allows; the
                    // thread's first kLinkRegs links keep their id, count,
                    // capacity left and share for the update
                    double sh = INFINITY;
                    uint32_t ll[kLinkRegs], lc[kLinkRegs];
                    double lr[kLinkRegs], ls[kLinkRegs];
#pragma unroll
                    for (uint32_t k = 0; k < kLinkRegs; ++k) {
                        const uint32_t i = tid + k * kSimThreads;
                        ll[k] = 0;
                        lc[k] = 0;
                        lr[k] = 0.0;
                        ls[k] = INFINITY;
                        if (i < nl) {
                            ll[k] = lk[i];
                            lc[k] = cnt[ll[k]];
                            if (lc[k] > 0) {
                                lr[k] = rem[ll[k]];
                                ls[k] = lr[k] / (double)lc[k];
                                sh = dmin(sh, ls[k]);
                            }
                        }
                    }
                    for (uint32_t i = tid + kLinkRegs * kSimThreads; i < nl; i += kSimThreads) {
                        const uint32_t l = lk[i];
                        const uint32_t c = cnt[l];
                        if (c > 0) sh = dmin(sh, rem[l] / (double)c);
                    }
                    const double inc = bmin(sh);
                    if (inc == INFINITY) break;
                    if (round > na) {   // every round freezes at least one flow
                        stall = 1;
                        break;
                    }
                    // links that the raise fills, and the capacity left on each
#pragma unroll
                    for (uint32_t k = 0; k < kLinkRegs; ++k) {
                        if (tid + k * kSimThreads < nl) {
                            uint8_t full = 0;
                            if (lc[k] > 0) {
                                full = ls[k] == inc ? 1 : 0;
                                const double used = inc * (double)lc[k];
                                const double lf = lr[k] - used;
                                rem[ll[k]] = lf > 0.0 ? lf : 0.0;
                            }
                            sat[ll[k]] = full;
                        }
                    }
                    for (uint32_t i = tid + kLinkRegs * kSimThreads; i < nl; i += kSimThreads) {
                        const uint32_t l = lk[i];
                        const uint32_t c = cnt[l];
                        uint8_t full = 0;
                        if (c > 0) {
                            const double r = rem[l];
                            full = r / (double)c == inc ? 1 : 0;
                            const double used = inc * (double)c;
                            const double lf = r - used;
                            rem[l] = lf > 0.0 ? lf : 0.0;
                        }
                        sat[l] = full;
                    }
                    level = level + inc;
                    __syncthreads();
                    // flows crossing a filled link stop at the current level
                    bool just = false;
                    if (!frozen) {
                        uint8_t hit = 0;
                        for (uint32_t u = 0; u < plen; ++u) hit |= sat[link(u)];
                        if (hit) {
                            just = true;
                            frozen = true;
                            rt = level;
                        }
                    }
                    if (just)
                        for (uint32_t u = 0; u < plen; ++u) atomicSub(&cnt[link(u)], 1u);
                    __syncthreads();
                    ++rounds;
                }
                if (stall) break;
                ++events;
                moving += na;
                // the next event: the earliest completion, or the next arrival
                const double dtc = bmin(has ? rm / rt : INFINITY);
                uint32_t nd = 0;
                if (dtc <= nx - t) {
                    if (has) {
                        if (rm / rt == dtc) {
                            a.state[f] = kDone;
                            a.finish[f] = t + dtc;
                            nd = 1;
                        } else {
                            const double moved = rt * dtc;
                            const double r = rm - moved;
                            a.remaining[f] = r > 0.0 ? r : 0.0;
                        }
                    }
                    t = t + dtc;
                } else {
                    const double dt = nx - t;
                    if (has) {
                        const double moved = rt * dt;
                        const double r = rm - moved;
                        a.remaining[f] = r > 0.0 ? r : 0.0;
                    }
                    t = nx;
                }
                left -= bsum(nd);
                continue;
            }
            // the max-min fair allocation of the moving flows: count them on
            // their links (a link's first count lists it and resets its capacity)
            for (uint32_t i = tid; i < na; i += kSimThreads) {
                const uint64_t f = f0 + mv[i];
                a.frz[f] = kFree;
                for (uint64_t q = a.path_off[f]; q < a.path_off[f + 1]; ++q) {
                    const uint32_t l = a.path[q];
                    if (atomicAdd(&cnt[l], 1u) == 0) {
                        rem[l] = LDS ? lcap[l] : cap[l];
                        lk[atomicAdd(&n_lk, 1u)] = l;
                    }
                }
            }
            __syncthreads();
            const uint32_t nl = n_lk;
            double level = 0.0;
            uint32_t unfrozen = na;
            for (uint32_t round = 0; unfrozen > 0; ++round) {
                if (round > na) {   // every round freezes at least one flow
                    stall = 1;
                    break;
                }
                // the largest equal raise every link still allows
                double sh = INFINITY;
                for (uint32_t i = tid; i < nl; i += kSimThreads) {
                    const uint32_t l = lk[i];
                    const uint32_t c = cnt[l];
                    if (c > 0) sh = dmin(sh, rem[l] / (double)c);
                }
                const double inc = bmin(sh);
                // links that the raise fills, and the capacity left on each
                for (uint32_t i = tid; i < nl; i += kSimThreads) {
                    const uint32_t l = lk[i];
                    const uint32_t c = cnt[l];
                    uint8_t full = 0;
                    if (c > 0) {
                        const double r = rem[l];
                        full = r / (double)c == inc ? 1 : 0;
                        const double used = inc * (double)c;
                        const double lf = r - used;
                        rem[l] = lf > 0.0 ? lf : 0.0;
                    }
                    sat[l] = full;
                }
                level = level + inc;
                __syncthreads();
                // flows crossing a filled link stop at the current level
                uint32_t nfz = 0;
                for (uint32_t i = tid; i < na; i += kSimThreads) {
                    const uint64_t f = f0 + mv[i];
                    if (a.frz[f] != kFree) continue;
                    uint8_t hit = 0;
                    for (uint64_t q = a.path_off[f]; q < a.path_off[f + 1]; ++q) hit |= sat[a.path[q]];
                    if (hit) {
                        a.frz[f] = kJustFrozen;
                        a.rate[f] = level;
                        ++nfz;
                    }
                }
                nfz = bsum(nfz);
                for (uint32_t i = tid; i < na; i += kSimThreads) {
                    const uint64_t f = f0 + mv[i];
                    if (a.frz[f] != kJustFrozen) continue;
                    a.frz[f] = kFrozen;
                    for (uint64_t q = a.path_off[f]; q < a.path_off[f + 1]; ++q) atomicSub(&cnt[a.path[q]], 1u);
                }
                __syncthreads();
                unfrozen -= nfz;
                ++rounds;
            }
            if (stall) break;
            ++events;
            moving += na;
            // the next event: the earliest completion, or the next arrival
            double tc = INFINITY;
            for (uint32_t i = tid; i < na; i += kSimThreads) {
                const uint64_t f = f0 + mv[i];
                tc = dmin(tc, a.remaining[f] / a.rate[f]);
            }
            const double dtc = bmin(tc);
            uint32_t nd = 0;
            if (dtc <= nx - t) {
                for (uint32_t i = tid; i < na; i += kSimThreads) {
                    const uint64_t f = f0 + mv[i];
                    const double rm = a.remaining[f], rt = a.rate[f];
                    if (rm / rt == dtc) {
                        a.state[f] = kDone;
                        a.finish[f] = t + dtc;
                        ++nd;
                    } else {
                        const double moved = rt * dtc;
                        const double r = rm - moved;
                        a.remaining[f] = r > 0.0 ? r : 0.0;
                    }
                }
                t = t + dtc;
            } else {
                const double dt = nx - t;
                for (uint32_t i = tid; i < na; i += kSimThreads) {
                    const uint64_t f = f0 + mv[i];
                    const double moved = a.rate[f] * dt;
                    const double r = a.remaining[f] - moved;
                    a.remaining[f] = r > 0.0 ? r : 0.0;
                }
                t = nx;
            }
            left -= bsum(nd);
        }
        if (tid == 0) {
            ctl.t = t;
            ctl.nx = nx;
            ctl.ap = ap;
            ctl.left = left;
            ctl.pass = pass;
            ctl.events = events;
            ctl.rounds = rounds;
            ctl.moving = moving;
            ctl.na = na;
            ctl.list = cur;
            ctl.mode = stall ? kRunEnd : next;
            ctl.resume = next == kRunWave ? 1u : 0u;
            ctl.stall = stall;
            n_lk = 0;
        }
        __syncthreads();
    }
    if (ctl.stall) {
        for (uint64_t f = f0 + tid; f < f1; f += kSimThreads)
            if (a.state[f] != kDone) a.finish[f] = NAN;
        if (tid == 0) atomicOr(a.err, kErrFlowStallBit);
    }
    if (tid == 0 && a.stats) {
        a.stats[3ull * inst + 0] = ctl.events;
        a.stats[3ull * inst + 1] = ctl.rounds;
        a.stats[3ull * inst + 2] = ctl.moving;
    }
}

// Whether flow_off partitions the call's flows (non-decreasing, ending at
// most at n_flows): *bad_off = 0 if so, else 1.  One workgroup.
__global__ __launch_bounds__(kSimThreads) void flow_check_kernel(const uint64_t *__restrict__ flow_off,
                                                                 uint32_t n_inst, uint64_t n_flows,
                                                                 uint32_t *__restrict__ bad_off) {
    __shared__ uint32_t any;
    if (threadIdx.x == 0) any = 0;
    __syncthreads();
    uint32_t b = 0;
    for (uint32_t i = threadIdx.x; i < n_inst; i += kSimThreads)
        if (flow_off[i] > flow_off[i + 1] || flow_off[i + 1] > n_flows) b = 1;
    if (b) atomicOr(&any, 1u);
    __syncthreads();
    if (threadIdx.x == 0) *bad_off = any;
}

// The arrival-order sort's input, one workgroup per instance: each flow's
// arrival time as a 64-bit key whose unsigned order is that of the times
// (the sign bit set on non-negative values, all bits inverted on negative
// ones), its offset in the instance as the value, and the instance's
// segment (empty for every instance when the offsets are invalid, so that
// the sort stays inside the flows).
// Per instance: the arrival-order sort's keys and segments, and the
// instance's weight for the launch order, the sum over its flows of bytes
// over the least capacity on the path (its rank agrees closely with the
// instance's count of filling rounds).  Instances share the CUs, and one
// holds the call until its last instance ends: workgroups taking the
// heaviest instances first spread them over the CUs, beside lighter ones.
// The weight skips what the simulation rejects (paths outside the path
// array, links past n_links, bytes that are negative or not finite), and is
// summed in a fixed order, so the launch order is the same for the same
// input; no instance's results depend on it.
__global__ __launch_bounds__(kSimThreads) void flow_keys_kernel(const uint64_t *__restrict__ flow_off,
                                                                const double *__restrict__ start,
                                                                const uint32_t *__restrict__ bad_off,
                                                                const double *__restrict__ cap, uint32_t n_links,
                                                                const uint64_t *__restrict__ path_off,
                                                                const uint32_t *__restrict__ path, uint64_t n_path,
                                                                const double *__restrict__ bytes,
                                                                uint64_t *__restrict__ keys,
                                                                uint32_t *__restrict__ vals,
                                                                uint32_t *__restrict__ seg_b,
                                                                uint32_t *__restrict__ seg_e,
                                                                uint32_t *__restrict__ wkey,
                                                                uint32_t *__restrict__ widx) {
    __shared__ double red[kSimThreads];
    const uint32_t inst = blockIdx.x;
    const bool ok = *bad_off == 0;
    const uint64_t f0 = ok ? flow_off[inst] : 0, f1 = ok ? flow_off[inst + 1] : 0;   // < 2^32 when ok
    if (threadIdx.x == 0) {
        seg_b[inst] = (uint32_t)f0;
        seg_e[inst] = (uint32_t)f1;
    }
    const double *c = cap + (uint64_t)inst * n_links;
    double w = 0.0;
    for (uint64_t f = f0 + threadIdx.x; f < f1; f += kSimThreads) {
        const uint64_t u = (uint64_t)__double_as_longlong(start[f]);
        keys[f] = (u >> 63) ? ~u : (u | (1ull << 63));
        vals[f] = (uint32_t)(f - f0);
        const uint64_t p0 = path_off[f], p1 = path_off[f + 1];
        double cm = __builtin_inf();
        if (p1 > p0 && p1 <= n_path)
            for (uint64_t q = p0; q < p1; ++q) {
                const uint32_t l = path[q];
                if (l < n_links) cm = fmin(cm, c[l]);
            }
        const double b = bytes[f];
        if (b >= 0.0 && isfinite(b) && cm > 0.0 && isfinite(cm)) w += b / cm;
    }
    red[threadIdx.x] = w;
    __syncthreads();
    for (uint32_t h = kSimThreads / 2; h > 0; h /= 2) {
        if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        // descending weight as an ascending key (a weight is >= 0, so its
        // fp32 bits grow with it)
        const float wf = (float)red[0];
        wkey[inst] = ~__float_as_uint(isfinite(wf) ? wf : 3.0e38f);
        widx[inst] = inst;
    }
}

inline uint64_t align256(uint64_t x) { return (x + 255) / 256 * 256; }

}  // namespace

extern "C" netkv_status netkv_flow_sim(netkv_handle h, uint32_t n_inst, uint32_t n_links, const double *cap,
                                       const uint64_t *flow_off, uint64_t n_flows, const uint64_t *path_off,
                                       const uint32_t *path, uint64_t n_path, const double *bytes,
                                       const double *start, double *finish, uint64_t *stats, void *stream) {
    if (!h) return NETKV_EINVAL;
    netkv_internal_clear(h);
    if (n_inst == 0) return NETKV_OK;
    if (n_links == 0) return netkv_internal_fail(h, NETKV_EINVAL, "n_links must be >= 1");
    if (n_inst > 0x7FFFFFFFu) return netkv_internal_fail(h, NETKV_EINVAL, "n_inst must be < 2^31");
    if (!cap || !flow_off || !path_off || (n_flows && (!bytes || !start || !finish)) || (n_path && !path))
        return netkv_internal_fail(h, NETKV_EINVAL, "NULL array");
    if (n_flows >= (1ull << 32) || n_path > (1ull << 40))
        return netkv_internal_fail(h, NETKV_EINVAL, "n_flows must be < 2^32 and n_path <= 2^40");
    const int dev = netkv_internal_device(h);
    int prev = -1;
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
    const bool lds = n_links <= kSimLdsLinks;
    hipStream_t s = (hipStream_t)stream;
    // the arrival-order sort: keys in `remaining` and values in the first
    // moving list (the simulation initialises both itself), the sorted keys
    // in `skey`, the order in `arr`
    size_t sort_bytes = 0;
    hipError_t e = hipSuccess;
    if (n_flows)
        e = rocprim::segmented_radix_sort_pairs(nullptr, sort_bytes, (const uint64_t *)nullptr, (uint64_t *)nullptr,
                                                (const uint32_t *)nullptr, (uint32_t *)nullptr, (unsigned)n_flows,
                                                n_inst, (const uint32_t *)nullptr, (const uint32_t *)nullptr, 0, 64, s);
    if (e != hipSuccess) {
        if (prev >= 0 && prev != dev) (void)hipSetDevice(prev);
        return netkv_internal_fail(h, NETKV_EDEVICE, "arrival sort size query failed");
    }
    // the launch order's sort of the instances' weights
    size_t isort_bytes = 0;
    if (e == hipSuccess && n_flows)
        e = rocprim::radix_sort_pairs(nullptr, isort_bytes, (const uint32_t *)nullptr, (uint32_t *)nullptr,
                                      (const uint32_t *)nullptr, (uint32_t *)nullptr, n_inst, 0, 32, s);
    if (e != hipSuccess) {
        if (prev >= 0 && prev != dev) (void)hipSetDevice(prev);
        return netkv_internal_fail(h, NETKV_EDEVICE, "launch-order sort size query failed");
    }
    const uint64_t per_flow = align256(8 * n_flows) * 3 + align256(n_flows) * 2 + align256(4 * n_flows) * 3;
    const uint64_t per_inst = 6 * align256(4ull * n_inst) + 256 + align256(sort_bytes) + align256(isort_bytes);
    const uint64_t per_link = lds ? 0 : align256(8ull * n_inst * n_links) + 2 * align256(4ull * n_inst * n_links) +
                                            align256((uint64_t)n_inst * n_links);
    void *buf = nullptr;
    netkv_status st = NETKV_OK;
    e = netkv_internal_flow_buffer(h, per_flow + per_inst + per_link + 256, &buf);
    if (e != hipSuccess) {
        st = netkv_internal_fail(h, e == hipErrorOutOfMemory ? NETKV_ENOMEM : NETKV_EDEVICE,
                                 "flow simulation work buffer allocation failed");
    } else {
        uint8_t *p = (uint8_t *)buf;
        SimArgs a{};
        a.n_links = n_links;
        a.cap = cap;
        a.flow_off = flow_off;
        a.n_flows = n_flows;
        a.path_off = path_off;
        a.path = path;
        a.n_path = n_path;
        a.bytes = bytes;
        a.start = start;
        a.finish = finish;
        a.stats = stats;
        a.remaining = (double *)p;
        p += align256(8 * n_flows);
        a.rate = (double *)p;
        p += align256(8 * n_flows);
        a.state = p;
        p += align256(n_flows);
        a.frz = p;
        p += align256(n_flows);
        a.mlist = (uint32_t *)p;
        p += align256(4 * n_flows);
        a.mlist2 = (uint32_t *)p;
        p += align256(4 * n_flows);
        uint32_t *arr = (uint32_t *)p;
        a.arr = arr;
        p += align256(4 * n_flows);
        uint64_t *skey = (uint64_t *)p;
        a.skey = skey;
        p += align256(8 * n_flows);
        uint32_t *seg_b = (uint32_t *)p;
        p += align256(4ull * n_inst);
        uint32_t *seg_e = (uint32_t *)p;
        p += align256(4ull * n_inst);
        uint32_t *bad_off = (uint32_t *)p;
        a.bad_off = bad_off;
        p += 256;
        void *sort_tmp = p;
        p += align256(sort_bytes);
        uint32_t *wkey = (uint32_t *)p;
        p += align256(4ull * n_inst);
        uint32_t *wkey2 = (uint32_t *)p;
        p += align256(4ull * n_inst);
        uint32_t *widx = (uint32_t *)p;
        p += align256(4ull * n_inst);
        uint32_t *order = (uint32_t *)p;
        p += align256(4ull * n_inst);
        void *isort_tmp = p;
        p += align256(isort_bytes);
        if (!lds) {
            a.g_rem = (double *)p;
            p += align256(8ull * n_inst * n_links);
            a.g_cnt = (uint32_t *)p;
            p += align256(4ull * n_inst * n_links);
            a.g_lk = (uint32_t *)p;
            p += align256(4ull * n_inst * n_links);
            a.g_sat = p;
        }
        a.err = netkv_internal_errword(h);
        hipLaunchKernelGGL(flow_check_kernel, dim3(1), dim3(kSimThreads), 0, s, flow_off, n_inst, n_flows, bad_off);
        if (n_flows) {
            hipLaunchKernelGGL(flow_keys_kernel, dim3(n_inst), dim3(kSimThreads), 0, s, flow_off, start,
                               (const uint32_t *)bad_off, cap, n_links, path_off, path, n_path, bytes,
                               (uint64_t *)a.remaining, a.mlist, seg_b, seg_e, wkey, widx);
            size_t tb = sort_bytes;
            e = rocprim::segmented_radix_sort_pairs(sort_tmp, tb, (const uint64_t *)a.remaining, skey,
                                                    (const uint32_t *)a.mlist, arr, (unsigned)n_flows, n_inst,
                                                    (const uint32_t *)seg_b, (const uint32_t *)seg_e, 0, 64, s);
            if (e == hipSuccess) {
                size_t ib = isort_bytes;
                e = rocprim::radix_sort_pairs(isort_tmp, ib, (const uint32_t *)wkey, wkey2, (const uint32_t *)widx,
                                              order, n_inst, 0, 32, s);
                a.order = order;
            }
        }
        if (e == hipSuccess && lds)
            hipLaunchKernelGGL(flow_sim_kernel<true>, dim3(n_inst), dim3(kSimThreads), lds_link_bytes(n_links), s, a);
        else if (e == hipSuccess)
            hipLaunchKernelGGL(flow_sim_kernel<false>, dim3(n_inst), dim3(kSimThreads), 0, s, a);
        if (e == hipSuccess) e = hipGetLastError();
        if (e != hipSuccess) st = netkv_internal_fail(h, NETKV_EDEVICE, hipGetErrorString(e));
    }
    if (prev >= 0 && prev != dev) (void)hipSetDevice(prev);
    return st;
}

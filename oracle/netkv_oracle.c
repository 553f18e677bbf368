/*
 * Plain CPU oracle for NetKV decode-instance selection.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no source, header, table or helper with the
 * HIP library: it has its own structures, its own resident-set structure
 * (a sorted copy of each decode's hash list, searched by bisection -- the
 * GPU path uses open-addressed tables instead) and computes in fp64.
 *
 * What it computes (paper: "NetKV: Network-Aware Decode Instance Selection
 * for Disaggregated LLM Inference"):
 *   - Sec. III-B: n_r = floor(l_r / B_tok) hashed blocks; the cache hit is
 *     B_tok times the number of leading blocks of h_r resident on d (the
 *     block-level longest common prefix, scanned up to the first miss).
 *   - Eq. (2): non-cached bytes s_eff = s_r (1 - lambda / l_r), evaluated in
 *     the algebraically identical integer form bpt * (l_r - lambda), with
 *     bpt the per-GPU-pair KV bytes per token of Eq. (1).
 *   - Eq. (4): B_eff = B_tau (1 - c) / (1 + n_inflight[tau][p]).
 *   - Eq. (3): T_transfer = s_eff / B_eff + L_tau.
 *   - Sec. IV-B, Eqs. (6)-(7): T_queue = max(0, q_d - (beta_max - beta_d)) t_iter(beta_d),
 *     T_decode = t_iter(beta_d + 1), t_iter(beta) = a + b beta (Sec. III-C).
 *   - Eq. (5) / Algorithm 1: feasible set m_d >= s_eff + m_min; cost
 *     C = T_transfer + alpha (T_queue + T_decode) (alpha = 1 is Eq. (5));
 *     select the minimum-cost feasible d, ties to the lowest index; reject
 *     (index -1, cost +inf) when no d is feasible.
 *   Every request is scored against the same snapshot (the in-flight counter
 *   update of Algorithm 1 happens between batches, see orc_commit).
 *
 * Readings where the paper is silent: congestion is given per (p, d) pair;
 * the block size is a parameter; all decodes are matched before the
 * feasibility filter.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    uint32_t n_prefill, n_decode;
    const uint8_t *tier_map;      /* [n_prefill * n_decode] */
    const float *util;            /* [n_prefill * n_decode] congestion c(p,d) */
    const uint16_t *n_inflight;   /* [4 * n_prefill], tier-major */
    double tier_bw[4];            /* bytes/s */
    double tier_lat[4];           /* s */
    const uint64_t *free_mem;     /* [n_decode] m_d, bytes */
    const uint32_t *queue_depth;  /* [n_decode] q_d */
    const uint32_t *batch_size;   /* [n_decode] beta_d */
    double t_iter_a, t_iter_b;
    uint32_t beta_max;
    double alpha;
    uint64_t m_min;
    uint64_t kv_bytes_per_token;
    uint32_t block_tokens;
    /* two-hop routing (Sec. VIII): the staged route p -> store -> d of every
     * pair, hop tiers and congestion [n_prefill * n_decode]; NULL: none */
    const uint8_t *route_tier1;
    const float *route_util1;
    const uint8_t *route_tier2;
    const float *route_util2;
} orc_snapshot;

typedef struct {
    uint32_t n_req;
    const uint32_t *prefill;
    const uint32_t *len_tokens;
    const uint64_t *hash_off;     /* [n_req + 1] */
    const uint64_t *hashes;
} orc_requests;

/* ---------------------------------------------------------------- cache */

typedef struct {
    uint32_t n_decode;
    uint64_t *off;      /* [n_decode + 1] */
    uint64_t *keys;     /* each decode's hashes, sorted ascending */
} orc_cache;

static int cmp_u64(const void *a, const void *b) {
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return (x > y) - (x < y);
}

orc_cache *orc_cache_build(uint32_t n_decode, const uint64_t *off, const uint64_t *hashes,
                           int n_threads) {
    orc_cache *c = (orc_cache *)calloc(1, sizeof(orc_cache));
    uint64_t total = off[n_decode];
    c->n_decode = n_decode;
    c->off = (uint64_t *)malloc(sizeof(uint64_t) * (n_decode + 1));
    c->keys = (uint64_t *)malloc(sizeof(uint64_t) * (total ? total : 1));
    memcpy(c->off, off, sizeof(uint64_t) * (n_decode + 1));
    memcpy(c->keys, hashes, sizeof(uint64_t) * total);
#ifdef _OPENMP
    if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads)
#endif
    for (int64_t d = 0; d < (int64_t)n_decode; ++d)
        qsort(c->keys + off[d], (size_t)(off[d + 1] - off[d]), sizeof(uint64_t), cmp_u64);
    (void)n_threads;
    return c;
}

void orc_cache_free(orc_cache *c) {
    if (!c) return;
    free(c->off);
    free(c->keys);
    free(c);
}

/* Is block hash h in K_d?  (bisection over the sorted copy) */
static int resident(const orc_cache *c, uint32_t d, uint64_t h) {
    const uint64_t *k = c->keys + c->off[d];
    uint64_t lo = 0, hi = c->off[d + 1] - c->off[d];
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        if (k[mid] < h) lo = mid + 1;
        else hi = mid;
    }
    return lo < c->off[d + 1] - c->off[d] && k[lo] == h;
}

/* |LCP_block(h_r, K_d)|: leading blocks resident on d, up to the first miss
 * (Sec. III-B).  *tests receives the number of membership tests made. */
static uint32_t prefix_blocks(const orc_cache *c, uint32_t d, const uint64_t *h, uint32_t n,
                              uint32_t *tests) {
    uint32_t j = 0;
    while (j < n && resident(c, d, h[j])) ++j;
    *tests = (j < n) ? j + 1 : n;
    return j;
}

/* ---------------------------------------------------------------- costs */

static double t_iter(const orc_snapshot *s, double beta) { return s->t_iter_a + s->t_iter_b * beta; }

/* T_queue(d) + T_decode(d), Sec. IV-B */
static double load_time(const orc_snapshot *s, uint32_t d) {
    int64_t q = s->queue_depth[d], beta = s->batch_size[d];
    int64_t blocked = q - ((int64_t)s->beta_max - beta);
    if (blocked < 0) blocked = 0;
    double tq = (double)blocked * t_iter(s, (double)beta);
    double tdec = t_iter(s, (double)(beta + 1));
    return tq + tdec;
}

/* Eq. (4) */
static double eff_bandwidth(const orc_snapshot *s, uint32_t p, uint32_t d) {
    uint64_t pd = (uint64_t)p * s->n_decode + d;
    int tau = s->tier_map[pd];
    double c = (double)s->util[pd];
    double n = (double)s->n_inflight[(uint64_t)tau * s->n_prefill + p];
    return s->tier_bw[tau] * (1.0 - c) / (1.0 + n);
}

/* Transfer time of s_eff bytes from p to d (Eq. (3)): the direct route, or
 * with staged routes the faster of the direct one and the sum of the two
 * hops' transfer times (Sec. VIII; the staging store's transfers carry no
 * in-flight count of the prefill).  *staged tells which (ties: direct). */
static double transfer_time(const orc_snapshot *s, uint32_t p, uint32_t d, uint64_t s_eff, int *staged) {
    uint64_t pd = (uint64_t)p * s->n_decode + d;
    int tau = s->tier_map[pd];
    double direct = (double)s_eff / eff_bandwidth(s, p, d) + s->tier_lat[tau];
    *staged = 0;
    if (!s->route_tier1) return direct;
    int t1 = s->route_tier1[pd], t2 = s->route_tier2[pd];
    double n1 = (double)s->n_inflight[(uint64_t)t1 * s->n_prefill + p];
    double b1 = s->tier_bw[t1] * (1.0 - (double)s->route_util1[pd]) / (1.0 + n1);
    double b2 = s->tier_bw[t2] * (1.0 - (double)s->route_util2[pd]);
    double two = (double)s_eff / b1 + s->tier_lat[t1] + (double)s_eff / b2 + s->tier_lat[t2];
    if (two < direct) {
        *staged = 1;
        return two;
    }
    return direct;
}

typedef struct {
    double cost;
    int32_t d;
} cand;

static int cmp_cand(const void *a, const void *b) {
    const cand *x = (const cand *)a, *y = (const cand *)b;
    if (x->cost < y->cost) return -1;
    if (x->cost > y->cost) return 1;
    return (x->d > y->d) - (x->d < y->d);
}

/* Score request r against every decode with the congestion matrix `util`
 * (the snapshot's own, or a scenario's).  j_row, if given, supplies the
 * prefix lengths instead of matching again. */
static void score_request(const orc_snapshot *s, const float *util, const orc_cache *c,
                          const orc_requests *q, uint32_t r, const uint32_t *j_row, cand *buf,
                          uint32_t k, int32_t *out_idx, double *out_score, uint32_t *pj,
                          uint8_t *pf, double *pc, uint64_t *tests_sum) {
    orc_snapshot sv = *s;
    sv.util = util;
    uint32_t p = q->prefill[r];
    uint64_t len = q->len_tokens[r];
    uint64_t a = q->hash_off[r], b = q->hash_off[r + 1];
    uint32_t n = (uint32_t)(b - a);
    uint32_t nfeas = 0;
    uint64_t tests_r = 0;
    for (uint32_t d = 0; d < s->n_decode; ++d) {
        uint32_t j, t = 0;
        if (j_row) {
            j = j_row[d];
        } else {
            j = prefix_blocks(c, d, q->hashes + a, n, &t);
            tests_r += t;
        }
        uint64_t lambda = (uint64_t)s->block_tokens * j;               /* tokens */
        uint64_t s_eff = s->kv_bytes_per_token * (len - lambda);       /* Eq. (2) */
        uint64_t m = s->free_mem[d];
        int feas = (m >= s->m_min) && (m - s->m_min >= s_eff);         /* m >= s_eff + m_min */
        int staged;
        double t_x = transfer_time(&sv, p, d, s_eff, &staged);              /* Eq. (3) */
        double cost = t_x + s->alpha * load_time(s, d);
        if (pj) pj[d] = j;
        if (pf) pf[d] = (uint8_t)feas;
        if (pc) pc[d] = cost;
        if (feas) {
            buf[nfeas].cost = cost;
            buf[nfeas].d = (int32_t)d;
            ++nfeas;
        }
    }
    qsort(buf, nfeas, sizeof(cand), cmp_cand);
    for (uint32_t i = 0; i < k; ++i) {
        out_idx[i] = i < nfeas ? buf[i].d : -1;
        out_score[i] = i < nfeas ? buf[i].cost : INFINITY;
    }
    *tests_sum += tests_r;
}

/* Select top-k decodes for every request.  Per-pair outputs (row-major
 * [n_req][n_decode]) may be NULL.  Returns the number of block membership
 * tests made by the first-miss scans (sum over pairs of min(j + 1, n_r)). */
uint64_t orc_select(const orc_snapshot *s, const orc_cache *c, const orc_requests *q, uint32_t k,
                    int32_t *out_idx, double *out_score, uint32_t *pair_j, uint8_t *pair_feas,
                    double *pair_cost, int n_threads) {
    uint64_t tests = 0;
    const uint32_t D = s->n_decode;
#ifdef _OPENMP
    if (n_threads < 1) n_threads = 1;
#pragma omp parallel num_threads(n_threads) reduction(+ : tests)
#endif
    {
        cand *buf = (cand *)malloc(sizeof(cand) * (D ? D : 1));
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 8)
#endif
        for (int64_t r = 0; r < (int64_t)q->n_req; ++r) {
            uint64_t row = (uint64_t)r * D;
            score_request(s, s->util, c, q, (uint32_t)r, NULL, buf, k, out_idx + (uint64_t)r * k,
                          out_score + (uint64_t)r * k, pair_j ? pair_j + row : NULL,
                          pair_feas ? pair_feas + row : NULL, pair_cost ? pair_cost + row : NULL,
                          &tests);
        }
        free(buf);
    }
    return tests;
}

/* Ranking sweep over telemetry scenarios.  The prefix lengths do not depend
 * on telemetry, so they are matched once and reused for every scenario.
 * For each scenario the top-k is written to out_idx/out_score
 * ([n_scen][n_req][k]); out_flips[2*s] counts requests whose selected
 * decode's tier differs from the tier selected under the snapshot's own
 * congestion, out_flips[2*s+1] those whose selected decode differs
 * (a rejection counts as its own tier and index). */
void orc_rank_sweep(const orc_snapshot *s_in, const orc_cache *c, const orc_requests *q,
                    uint32_t n_scen, const float *util_scen, uint32_t k, int32_t *out_idx,
                    double *out_score, uint64_t *out_flips, int n_threads) {
    orc_snapshot sd = *s_in;
    sd.route_tier1 = NULL;   /* the ranking sweep scores direct routes */
    const orc_snapshot *s = &sd;
    const uint32_t D = s->n_decode, R = q->n_req;
    uint32_t *jm = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)R * (D ? D : 1));
    int32_t *base = (int32_t *)malloc(sizeof(int32_t) * (R ? R : 1));
#ifdef _OPENMP
    if (n_threads < 1) n_threads = 1;
#pragma omp parallel num_threads(n_threads)
#endif
    {
        cand *buf = (cand *)malloc(sizeof(cand) * (D ? D : 1));
        int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (k ? k : 1));
        double *sc = (double *)malloc(sizeof(double) * (k ? k : 1));
        uint64_t dummy = 0;
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 8)
#endif
        for (int64_t r = 0; r < (int64_t)R; ++r) {
            score_request(s, s->util, c, q, (uint32_t)r, NULL, buf, 1, idx, sc,
                          jm + (uint64_t)r * D, NULL, NULL, &dummy);
            base[r] = idx[0];
        }
        free(buf);
        free(idx);
        free(sc);
    }
    for (uint32_t sn = 0; sn < n_scen; ++sn) {
        const float *u = util_scen + (uint64_t)sn * s->n_prefill * D;
        uint64_t tier_flips = 0, idx_flips = 0;
#ifdef _OPENMP
#pragma omp parallel num_threads(n_threads) reduction(+ : tier_flips, idx_flips)
#endif
        {
            cand *buf = (cand *)malloc(sizeof(cand) * (D ? D : 1));
            uint64_t dummy = 0;
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 8)
#endif
            for (int64_t r = 0; r < (int64_t)R; ++r) {
                uint64_t o = ((uint64_t)sn * R + (uint64_t)r) * k;
                score_request(s, u, c, q, (uint32_t)r, jm + (uint64_t)r * D, buf, k, out_idx + o,
                              out_score + o, NULL, NULL, NULL, &dummy);
                int32_t a = base[r], b = out_idx[o];
                uint32_t p = q->prefill[r];
                int ta = a < 0 ? -1 : s->tier_map[(uint64_t)p * D + (uint32_t)a];
                int tb = b < 0 ? -1 : s->tier_map[(uint64_t)p * D + (uint32_t)b];
                tier_flips += (ta != tb);
                idx_flips += (a != b);
            }
            free(buf);
        }
        if (out_flips) {
            out_flips[2 * sn] = tier_flips;
            out_flips[2 * sn + 1] = idx_flips;
        }
    }
    free(jm);
    free(base);
}

/* Proposition 2 (Sec. V-D): tier-ranking inversions under a congestion
 * scenario.  For every prefill instance p and every pair of decodes d, d'
 * on different tiers from p, the bandwidths of Eq. (4) are compared under
 * the loaded snapshot's congestion c and under the scenario's c^:
 *     X = B'_tau (1 - c),  B'_tau = B_tau / (1 + n_inflight[tau][p])
 * (the proposition states n = 0; the in-flight count is the same in both,
 * so it scales B_tau only).  A pair whose snapshot values differ is
 * inverted when the scenario does not keep that strict order.  The
 * proposition's sufficient condition, taken per pair: with
 *     eps = max(|c^(p,d) - c(p,d)|, |c^(p,d') - c(p,d')|),
 * the order is kept when eps < |X - X'| / (B'_tau + B'_tau').  Per scenario
 * out[3s + 0] = pairs the condition covers, out[3s + 1] = inverted pairs
 * among them (0 by the proposition), out[3s + 2] = all inverted pairs.
 * Every quantity is evaluated in fp64 in exactly this order:
 *     b = tier_bw[tau] / (1.0 + n);  X = b * (1.0 - (double)c);
 *     bound = |X - X'| / (b + b');   eps from the exact float differences. */
static double share_bw(const orc_snapshot *s, uint32_t p, int tau) {
    return s->tier_bw[tau] / (1.0 + (double)s->n_inflight[(uint64_t)tau * s->n_prefill + p]);
}

void orc_tier_inversions(const orc_snapshot *s, uint32_t n_scen, const float *util_scen, uint64_t *out,
                         int n_threads) {
    const uint32_t P = s->n_prefill, D = s->n_decode;
    for (uint32_t sn = 0; sn < n_scen; ++sn) {
        const float *u = util_scen + (uint64_t)sn * P * D;
        uint64_t covered = 0, inv_covered = 0, inverted = 0;
#ifdef _OPENMP
        if (n_threads < 1) n_threads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads) reduction(+ : covered, inv_covered, inverted)
#endif
        for (int64_t p = 0; p < (int64_t)P; ++p) {
            for (uint32_t d = 0; d < D; ++d) {
                const uint64_t a = (uint64_t)p * D + d;
                const int ta = s->tier_map[a];
                const double ba = share_bw(s, (uint32_t)p, ta);
                const double ca = (double)s->util[a], ha = (double)u[a];
                const double xa = ba * (1.0 - ca), ya = ba * (1.0 - ha);
                for (uint32_t e = d + 1; e < D; ++e) {
                    const uint64_t b = (uint64_t)p * D + e;
                    const int tb = s->tier_map[b];
                    if (tb == ta) continue;   /* only pairs across tiers */
                    const double bb = share_bw(s, (uint32_t)p, tb);
                    const double cb = (double)s->util[b], hb = (double)u[b];
                    const double xb = bb * (1.0 - cb), yb = bb * (1.0 - hb);
                    if (xa == xb) continue;   /* no strict order to keep */
                    const int inv = xa > xb ? !(ya > yb) : !(ya < yb);
                    const double eps = fmax(fabs(ha - ca), fabs(hb - cb));
                    const int cov = eps < fabs(xa - xb) / (ba + bb);
                    covered += (uint64_t)cov;
                    inv_covered += (uint64_t)(cov && inv);
                    inverted += (uint64_t)inv;
                }
            }
        }
        out[3 * (uint64_t)sn] = covered;
        out[3 * (uint64_t)sn + 1] = inv_covered;
        out[3 * (uint64_t)sn + 2] = inverted;
    }
    (void)n_threads;
}

/* State carried from one batch to the next (streaming workload).
 * Algorithm 1 increments n_inflight[tau(p, d*)][p] after each selection and
 * the paper caps the counter (default 16); the transfer-complete callback
 * decrements it.  Reading used here, with one batch as the unit of time:
 * transfers of earlier batches have completed, so after a batch
 *   n_inflight[tau][p] = min(cap, #selections of the batch from p on tau);
 * each decode serves up to `mu` queued requests per batch interval,
 *   q_d = max(0, q_d + admitted_d - mu);
 * the KV bytes admitted in this batch occupy decode memory until the next
 * batch completes them,
 *   m_d = max(0, m_d - A_d) + A_prev_d,   A_prev_d <- A_d,
 * with A_d the sum of s_eff over the requests admitted to d.
 * All of it is integer arithmetic. */
void orc_commit(const orc_snapshot *s, const orc_cache *c, const orc_requests *q,
                const int32_t *sel, uint32_t cap, uint32_t mu, uint16_t *n_inflight,
                uint32_t *queue_depth, uint64_t *free_mem, uint64_t *admitted_prev) {
    const uint32_t P = s->n_prefill, D = s->n_decode;
    uint64_t *cnt = (uint64_t *)calloc((size_t)4 * P, sizeof(uint64_t));
    uint64_t *adm = (uint64_t *)calloc(D ? D : 1, sizeof(uint64_t));
    uint64_t *bytes = (uint64_t *)calloc(D ? D : 1, sizeof(uint64_t));
    for (uint32_t r = 0; r < q->n_req; ++r) {
        int32_t d = sel[r];
        if (d < 0) continue;
        uint32_t p = q->prefill[r];
        int tau = s->tier_map[(uint64_t)p * D + (uint32_t)d];
        uint32_t t;
        uint64_t a = q->hash_off[r];
        uint32_t n = (uint32_t)(q->hash_off[r + 1] - a);
        uint32_t j = prefix_blocks(c, (uint32_t)d, q->hashes + a, n, &t);
        uint64_t s_eff = s->kv_bytes_per_token * ((uint64_t)q->len_tokens[r] - (uint64_t)s->block_tokens * j);
        cnt[(uint64_t)tau * P + p] += 1;
        adm[d] += 1;
        bytes[d] += s_eff;
    }
    for (uint64_t i = 0; i < (uint64_t)4 * P; ++i) n_inflight[i] = (uint16_t)(cnt[i] < cap ? cnt[i] : cap);
    for (uint32_t d = 0; d < D; ++d) {
        int64_t nq = (int64_t)queue_depth[d] + (int64_t)adm[d] - (int64_t)mu;
        queue_depth[d] = (uint32_t)(nq < 0 ? 0 : nq);
        uint64_t m = free_mem[d];
        m = (m > bytes[d]) ? m - bytes[d] : 0;
        free_mem[d] = m + admitted_prev[d];
        admitted_prev[d] = bytes[d];
    }
    free(cnt);
    free(adm);
    free(bytes);
}

/* Algorithm 1 request by request, in batch order: each request is scored
 * with the in-flight counters left by the earlier requests (Algorithm 1
 * increments n_inflight[tau(p, d*)][p] after every selection; Sec. V-C caps
 * the counter, read here as a saturating increment: n < cap ? n + 1 : n).
 * out_idx/out_score receive each request's argmin.  If `follow` is not NULL
 * the counters advance with follow[r] instead of the oracle's own choice
 * (so a comparison can continue from another implementation's choices), and
 * follow_cost[r] receives the cost of follow[r] under the same counters
 * (+inf for -1, NaN when follow[r] is not a feasible decode). */
void orc_select_sequential(const orc_snapshot *s, const orc_cache *c, const orc_requests *q, uint32_t cap,
                           const int32_t *follow, int32_t *out_idx, double *out_score, double *follow_cost) {
    const uint32_t P = s->n_prefill, D = s->n_decode;
    uint16_t *n = (uint16_t *)malloc(sizeof(uint16_t) * 4 * (size_t)P);
    memcpy(n, s->n_inflight, sizeof(uint16_t) * 4 * (size_t)P);
    cand *buf = (cand *)malloc(sizeof(cand) * (D ? D : 1));
    uint8_t *feas = (uint8_t *)malloc(D ? D : 1);
    double *cost = (double *)malloc(sizeof(double) * (D ? D : 1));
    orc_snapshot sv = *s;
    sv.n_inflight = n;
    sv.route_tier1 = NULL;   /* the sequential form scores direct routes */
    for (uint32_t r = 0; r < q->n_req; ++r) {
        uint64_t tests = 0;
        score_request(&sv, s->util, c, q, r, NULL, buf, 1, out_idx + r, out_score + r, NULL, feas, cost, &tests);
        int32_t take = follow ? follow[r] : out_idx[r];
        if (follow_cost) {
            if (take < 0) follow_cost[r] = INFINITY;
            else if ((uint32_t)take < D && feas[take]) follow_cost[r] = cost[take];
            else follow_cost[r] = NAN;
        }
        if (take >= 0 && (uint32_t)take < D) {
            uint32_t p = q->prefill[r];
            int tau = s->tier_map[(uint64_t)p * D + (uint32_t)take];
            uint16_t *cnt = &n[(uint64_t)tau * P + p];
            if (*cnt < cap) *cnt += 1;
        }
    }
    free(n);
    free(buf);
    free(feas);
    free(cost);
}

/* Two-hop routing: for each selection idx[r*k+q] >= 0, out[r*k+q] = 1 when
 * its staged route is strictly faster than the direct one, else 0; -1 for
 * no selection. */
void orc_route_of(const orc_snapshot *s, const orc_cache *c, const orc_requests *q, uint32_t k,
                  const int32_t *idx, int8_t *out) {
    for (uint32_t r = 0; r < q->n_req; ++r) {
        uint64_t a = q->hash_off[r];
        uint32_t n = (uint32_t)(q->hash_off[r + 1] - a);
        for (uint32_t i = 0; i < k; ++i) {
            int32_t d = idx[(uint64_t)r * k + i];
            if (d < 0) {
                out[(uint64_t)r * k + i] = -1;
                continue;
            }
            uint32_t t;
            uint32_t j = prefix_blocks(c, (uint32_t)d, q->hashes + a, n, &t);
            uint64_t s_eff = s->kv_bytes_per_token * (q->len_tokens[r] - (uint64_t)s->block_tokens * j);
            int staged;
            (void)transfer_time(s, q->prefill[r], (uint32_t)d, s_eff, &staged);
            out[(uint64_t)r * k + i] = (int8_t)staged;
        }
    }
}

/* Eq. (2): the non-cached bytes s_eff = bpt * (l_r - B_tok * j) of each
 * selection idx[r*k + i] (0 for no selection): the size of the KV transfer
 * it starts. */
void orc_selection_bytes(const orc_snapshot *s, const orc_cache *c, const orc_requests *q, uint32_t k,
                         const int32_t *idx, uint64_t *out) {
    for (uint32_t r = 0; r < q->n_req; ++r) {
        uint64_t a = q->hash_off[r];
        uint32_t n = (uint32_t)(q->hash_off[r + 1] - a);
        for (uint32_t i = 0; i < k; ++i) {
            int32_t d = idx[(uint64_t)r * k + i];
            if (d < 0) {
                out[(uint64_t)r * k + i] = 0;
                continue;
            }
            uint32_t t;
            uint32_t j = prefix_blocks(c, (uint32_t)d, q->hashes + a, n, &t);
            out[(uint64_t)r * k + i] = s->kv_bytes_per_token * (q->len_tokens[r] - (uint64_t)s->block_tokens * j);
        }
    }
}

/* Requests per tier of the selected decode; counts[4] = rejected. */
void orc_tier_counts(const orc_snapshot *s, const orc_requests *q, const int32_t *sel, uint64_t *counts) {
    for (int t = 0; t < 5; ++t) counts[t] = 0;
    for (uint32_t r = 0; r < q->n_req; ++r) {
        if (sel[r] < 0) counts[4] += 1;
        else counts[s->tier_map[(uint64_t)q->prefill[r] * s->n_decode + (uint32_t)sel[r]]] += 1;
    }
}

/* Predictive congestion (Sec. VIII, reading: simple exponential smoothing
 * of the congestion telemetry): one step c <- c + beta (obs - c) per entry,
 * in fp64.  An observation outside [0, 1) or NaN leaves its entry as it
 * was.  Returns the number of such observations. */
uint64_t orc_smooth(double *c, const float *obs, uint64_t n, double beta) {
    uint64_t bad = 0;
    for (uint64_t i = 0; i < n; ++i) {
        const double o = (double)obs[i];
        if (!(o >= 0.0 && o < 1.0)) {
            bad += 1;
            continue;
        }
        c[i] = c[i] + beta * (o - c[i]);
    }
    return bad;
}

/* The first-miss prefix length of one hash run against one decode's set
 * (exposed for tests). */
uint32_t orc_prefix_len(const orc_cache *c, uint32_t d, const uint64_t *h, uint32_t n) {
    uint32_t t;
    return prefix_blocks(c, d, h, n, &t);
}

int orc_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------
 * Flow-level transfer simulation (Sec. VI-B, the evaluation simulator's
 * network model): KV transfers are flows over the links of their path; the
 * links are shared max-min fairly among the flows crossing them, and every
 * flow arrival or completion re-evaluates the allocation of all flows in
 * progress.  Background traffic is a steady utilisation already taken out
 * of each link's capacity by the caller (the mean-field model).  The paper
 * gives no algorithm; the allocation is the max-min fair one, computed by
 * progressive filling (Bertsekas & Gallager, "Data Networks", Sec. 6.5.2):
 * all unfrozen flows' rates rise together until some link is full; the
 * flows crossing a full link are frozen at that rate; repeat.  fp64, with
 * every operation written out in order (no contraction: the file is built
 * without FMA), so that a second implementation doing the same operations
 * gets the same bits.
 * ------------------------------------------------------------------------ */

typedef struct {
    uint32_t n_links;
    const double *cap;          /* [n_links] bytes/s available to the flows, > 0 */
    uint32_t n_flows;
    const uint64_t *path_off;   /* [n_flows + 1] */
    const uint32_t *path;       /* links of each flow (distinct within a flow, at least one) */
    const double *bytes;        /* [n_flows] bytes to move, >= 0 */
    const double *start;        /* [n_flows] arrival time, s */
} orc_flows;

/* Max-min fair rates of the flows with active[f] != 0 (others get 0).
 * Returns the number of filling rounds. */
uint32_t orc_maxmin(const orc_flows *F, const uint8_t *active, double *rate) {
    const uint32_t L = F->n_links, N = F->n_flows;
    double *rem = (double *)malloc(sizeof(double) * (L ? L : 1));
    uint32_t *cnt = (uint32_t *)calloc(L ? L : 1, sizeof(uint32_t));
    uint8_t *sat = (uint8_t *)malloc(L ? L : 1);
    uint8_t *frozen = (uint8_t *)calloc(N ? N : 1, 1);
    uint32_t unfrozen = 0, rounds = 0;
    for (uint32_t l = 0; l < L; ++l) rem[l] = F->cap[l];
    for (uint32_t f = 0; f < N; ++f) {
        rate[f] = 0.0;
        if (!active[f]) continue;
        ++unfrozen;
        for (uint64_t q = F->path_off[f]; q < F->path_off[f + 1]; ++q) cnt[F->path[q]] += 1;
    }
    double level = 0.0;
    while (unfrozen > 0) {
        /* the largest equal raise every link still allows */
        double inc = INFINITY;
        for (uint32_t l = 0; l < L; ++l)
            if (cnt[l] > 0) {
                const double share = rem[l] / (double)cnt[l];
                if (share < inc) inc = share;
            }
        /* links that the raise fills, and the capacity left on each */
        for (uint32_t l = 0; l < L; ++l) {
            sat[l] = 0;
            if (cnt[l] > 0) {
                sat[l] = rem[l] / (double)cnt[l] == inc;
                const double used = inc * (double)cnt[l];
                const double left = rem[l] - used;
                rem[l] = left > 0.0 ? left : 0.0;
            }
        }
        level = level + inc;
        /* flows crossing a filled link stop at the current level */
        for (uint32_t f = 0; f < N; ++f) {
            if (!active[f] || frozen[f]) continue;
            int hit = 0;
            for (uint64_t q = F->path_off[f]; q < F->path_off[f + 1]; ++q) hit |= sat[F->path[q]];
            if (hit) {
                frozen[f] = 2;   /* frozen this round */
                rate[f] = level;
                --unfrozen;
            }
        }
        for (uint32_t f = 0; f < N; ++f)
            if (frozen[f] == 2) {
                frozen[f] = 1;
                for (uint64_t q = F->path_off[f]; q < F->path_off[f + 1]; ++q) cnt[F->path[q]] -= 1;
            }
        ++rounds;
    }
    free(rem);
    free(cnt);
    free(sat);
    free(frozen);
    return rounds;
}

/* Event-driven simulation: flows start at their arrival time; between
 * events every flow in progress moves at its max-min fair rate; the next
 * event is the earliest completion (remaining / rate) or the next arrival.
 * finish[f] = the completion time of flow f.  stats (may be NULL) =
 * {allocations computed, filling rounds over all of them, flows in
 * progress summed over all of them}.  Returns the number of allocations. */
uint64_t orc_flow_sim(const orc_flows *F, double *finish, uint64_t *stats) {
    const uint32_t N = F->n_flows;
    uint8_t *state = (uint8_t *)calloc(N ? N : 1, 1);   /* 0 waiting, 1 in progress, 2 done */
    uint8_t *active = (uint8_t *)calloc(N ? N : 1, 1);
    double *remaining = (double *)malloc(sizeof(double) * (N ? N : 1));
    double *rate = (double *)malloc(sizeof(double) * (N ? N : 1));
    uint64_t events = 0, rounds = 0, moving = 0;
    uint32_t left = N;
    for (uint32_t f = 0; f < N; ++f) remaining[f] = F->bytes[f];
    double t = INFINITY;
    for (uint32_t f = 0; f < N; ++f)
        if (F->start[f] < t) t = F->start[f];
    while (left > 0) {
        uint32_t n_act = 0;
        for (uint32_t f = 0; f < N; ++f) {
            if (state[f] == 0 && F->start[f] <= t) state[f] = 1;
            active[f] = state[f] == 1;
            n_act += active[f];
        }
        double next = INFINITY;   /* the next arrival */
        for (uint32_t f = 0; f < N; ++f)
            if (state[f] == 0 && F->start[f] < next) next = F->start[f];
        if (n_act == 0) {
            t = next;
            continue;
        }
        rounds += orc_maxmin(F, active, rate);
        moving += n_act;
        ++events;
        double dtc = INFINITY;    /* the earliest completion from t */
        for (uint32_t f = 0; f < N; ++f)
            if (active[f]) {
                const double tf = remaining[f] / rate[f];
                if (tf < dtc) dtc = tf;
            }
        if (dtc <= next - t) {
            for (uint32_t f = 0; f < N; ++f) {
                if (!active[f]) continue;
                if (remaining[f] / rate[f] == dtc) {
                    state[f] = 2;
                    finish[f] = t + dtc;
                    --left;
                } else {
                    const double moved = rate[f] * dtc;
                    const double r = remaining[f] - moved;
                    remaining[f] = r > 0.0 ? r : 0.0;
                }
            }
            t = t + dtc;
        } else {
            const double dt = next - t;
            for (uint32_t f = 0; f < N; ++f) {
                if (!active[f]) continue;
                const double moved = rate[f] * dt;
                const double r = remaining[f] - moved;
                remaining[f] = r > 0.0 ? r : 0.0;
            }
            t = next;
        }
    }
    free(state);
    free(active);
    free(remaining);
    free(rate);
    if (stats) {
        stats[0] = events;
        stats[1] = rounds;
        stats[2] = moving;
    }
    return events;
}

/* ------------------------------------------------------------------------
 * Telemetry derivations (the operator's side of the interface): what the
 * snapshot's congestion map is made of.  These restate the readings that
 * the synthetic inputs follow, so that the inputs can be checked against
 * them.
 * ------------------------------------------------------------------------ */

/* Per-link utilisation to one congestion value per (p, d) pair (Sec. III-E
 * gives one congestion value per tier; reading: the snapshot carries one per
 * pair).  The pair's tier is the lowest level its two GPUs share: 0 same
 * node, 1 same leaf, 2 same pod, 3 otherwise.  Its congestion is the larger
 * utilisation of the two tier-level links at its ends: u0 per node (the
 * node's fabric), u1 per node (its NIC uplink), u2 per leaf (leaf-spine),
 * u3 per pod (pod-core); domain of tier 0 and 1 = node, 2 = leaf, 3 = pod.
 * Coordinates per prefill and per decode: node, leaf, pod indices.  Writes
 * tier [P*D] and util [P*D] (fp32 of the fp64 maximum). */
void orc_pair_congestion(uint32_t P, uint32_t D, const uint32_t *p_node, const uint32_t *p_leaf,
                         const uint32_t *p_pod, const uint32_t *d_node, const uint32_t *d_leaf,
                         const uint32_t *d_pod, const double *u0, const double *u1, const double *u2,
                         const double *u3, uint8_t *tier, float *util) {
    for (uint32_t p = 0; p < P; ++p)
        for (uint32_t d = 0; d < D; ++d) {
            uint8_t t;
            double a, b;
            if (p_node[p] == d_node[d]) {
                t = 0;
                a = u0[p_node[p]];
                b = u0[d_node[d]];
            } else if (p_leaf[p] == d_leaf[d]) {
                t = 1;
                a = u1[p_node[p]];
                b = u1[d_node[d]];
            } else if (p_pod[p] == d_pod[d]) {
                t = 2;
                a = u2[p_leaf[p]];
                b = u2[d_leaf[d]];
            } else {
                t = 3;
                a = u3[p_pod[p]];
                b = u3[d_pod[d]];
            }
            tier[(uint64_t)p * D + d] = t;
            util[(uint64_t)p * D + d] = (float)(a > b ? a : b);
        }
}

/* One AR(1) step of n link utilisations (reading of the streaming
 * workload's telemetry): next = clamp(mean + rho (cur - mean) + sigma eps,
 * 0, 0.99), with mean the link's initial utilisation and eps a standard
 * normal draw per link (given). */
void orc_ar1_step(uint64_t n, const double *cur, const double *mean, const double *eps, double rho,
                  double sigma, double *next) {
    for (uint64_t i = 0; i < n; ++i) {
        const double dev = cur[i] - mean[i];
        const double pull = rho * dev;
        const double shock = sigma * eps[i];
        double v = mean[i] + pull;
        v = v + shock;
        if (v < 0.0) v = 0.0;
        if (v > 0.99) v = 0.99;
        next[i] = v;
    }
}

/* Noisy telemetry of one scenario (Sec. V-D's stale congestion, reading:
 * lognormal noise): each link utilisation times exp(sigma z), z a standard
 * normal draw per link (given), capped at 0.99. */
void orc_link_noise(uint64_t n, const double *u, const double *z, double sigma, double *out) {
    for (uint64_t i = 0; i < n; ++i) {
        const double m = exp(sigma * z[i]);
        const double v = u[i] * m;
        out[i] = v < 0.99 ? v : 0.99;
    }
}

/*
 * Oracle: fp64 single-threaded flow-level simulator (CPU).
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this file's library; the simulator library and its
 * GPU kernels share no code with it.
 *
 * What it computes (Section 4.1, netsim; Section 4.2, the paragraph on the
 * network simulator with time rollback): flows of given sizes are released
 * over links of given capacities; between consecutive events every flow
 * keeps a constant rate; the rates are the max-min fair (per-flow fairness)
 * allocation of the active flows, found by progressive filling
 * (water-filling: find the bottleneck, give its flows their share, repeat).
 * The output is every flow's completion time.
 *
 * Rate solve, over the active set U with paths P_f and capacities c_l:
 *   R_l = c_l, n_l = #{f in U : l in P_f}
 *   repeat while U is not empty:
 *     s_l = R_l / n_l for every link with n_l > 0;  s* = min_l s_l
 *     B   = {l : n_l > 0, s_l <= s* * THR}           (THR = 1 + 1e-12)
 *     every f in U crossing a link of B gets r_f = s* and leaves U;
 *     k_l = number of such flows on l;  R_l = R_l - k_l*s*;  n_l -= k_l
 * Event loop, starting at t = 0:
 *   t_next = min(earliest pending release, min over active f of t + rem_f/r_f)
 *   flows with t + rem_f/r_f <= t_next*THR send their last byte at t_next and
 *   finish their path latency lat_f later (lat = NULL: zero); the others
 *   lose r_f*(t_next - t) bytes; t = t_next; a flow whose predecessors have
 *   all finished is released at start_f + (latest predecessor finish);
 *   released flows with release <= t arrive (zero-byte flows finish at once
 *   and release their successors, to a fixpoint); if the active set
 *   changed, solve again.
 *
 * The solve keeps links in a binary heap keyed by s_l and, per iteration,
 * visits only the flows of the bottleneck links; every s_l, k_l, R_l and
 * n_l value is the one the sweep form above produces (same operations,
 * same order per link), so the rates are identical bit for bit.
 * Build with -ffp-contract=off: every product and sum is rounded on its own.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define THR 1.000000000001

enum { OR_OK = 0, OR_INVALID = -1, OR_NOMEM = -2, OR_INTERNAL = -3, OR_LIMIT = -5 };
enum { WAITING = 0, PENDING = 1, ACTIVE = 2, DONE = 3 };

typedef struct { double key; int64_t id; int64_t ver; } item;
typedef struct { item* a; int64_t n, cap; } heap;

static int heap_push(heap* h, double key, int64_t id, int64_t ver) {
    if (h->n == h->cap) {
        int64_t nc = h->cap ? 2 * h->cap : 1024;
        item* na = (item*)realloc(h->a, (size_t)nc * sizeof(item));
        if (!na) return OR_NOMEM;
        h->a = na; h->cap = nc;
    }
    int64_t i = h->n++;
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (h->a[p].key <= key) break;
        h->a[i] = h->a[p];
        i = p;
    }
    h->a[i].key = key; h->a[i].id = id; h->a[i].ver = ver;
    return OR_OK;
}

static item heap_pop(heap* h) {
    item top = h->a[0];
    item last = h->a[--h->n];
    int64_t i = 0;
    for (;;) {
        int64_t c = 2 * i + 1;
        if (c >= h->n) break;
        if (c + 1 < h->n && h->a[c + 1].key < h->a[c].key) c++;
        if (last.key <= h->a[c].key) break;
        h->a[i] = h->a[c];
        i = c;
    }
    if (h->n > 0) h->a[i] = last;
    return top;
}

typedef struct {
    int64_t L, F;
    const double* cap;
    const int64_t* poff;
    const int32_t* plink;
    /* link -> flow incidence (transpose of the paths) */
    int64_t* lf_off;
    int64_t* lf_ids;
    /* per-link solve state */
    double* R;
    int64_t* n;
    int64_t* k;
    int64_t* ver;
    int64_t* stamp;
    int64_t* touched;
    int64_t* klist;
    int64_t* blist;
    /* per-flow */
    uint8_t* state;
    int64_t* frozen_at;
    double* rate;
    heap lheap;
    int64_t solve_id;
    int64_t iterations, flows_swept, inc_swept;
} solver;

/* Max-min rates of the flows in act[0..na) (all in state ACTIVE). */
static int solve(solver* S, const int64_t* act, int64_t na) {
    const int64_t sid = ++S->solve_id;
    int64_t nt = 0, nnz_u = 0;
    for (int64_t q = 0; q < na; q++) {
        int64_t f = act[q];
        for (int64_t e = S->poff[f]; e < S->poff[f + 1]; e++) {
            int64_t l = S->plink[e];
            if (S->stamp[l] != sid) {
                S->stamp[l] = sid;
                S->R[l] = S->cap[l];
                S->n[l] = 0;
                S->k[l] = 0;
                S->touched[nt++] = l;
            }
            S->n[l] += 1;
        }
        nnz_u += S->poff[f + 1] - S->poff[f];
    }
    S->lheap.n = 0;
    for (int64_t q = 0; q < nt; q++) {
        int64_t l = S->touched[q];
        S->ver[l] += 1;
        if (heap_push(&S->lheap, S->R[l] / (double)S->n[l], l, S->ver[l])) return OR_NOMEM;
    }
    int64_t unfrozen = na;
    while (unfrozen > 0) {
        /* s* = smallest current share */
        while (S->lheap.n > 0 && S->lheap.a[0].ver != S->ver[S->lheap.a[0].id]) heap_pop(&S->lheap);
        if (S->lheap.n == 0) return OR_INTERNAL;
        const double sstar = S->lheap.a[0].key;
        if (!(sstar > 0.0)) return OR_INTERNAL;
        const double thr = sstar * THR;
        S->iterations += 1;
        S->flows_swept += unfrozen;
        S->inc_swept += nnz_u;
        /* bottleneck set B: every current share <= s* * THR */
        int64_t nb = 0;
        while (S->lheap.n > 0) {
            item top = S->lheap.a[0];
            if (top.ver != S->ver[top.id]) { heap_pop(&S->lheap); continue; }
            if (!(top.key <= thr)) break;
            heap_pop(&S->lheap);
            S->blist[nb++] = top.id;
        }
        /* freeze every unfrozen flow that crosses B at rate s* */
        int64_t nk = 0;
        for (int64_t b = 0; b < nb; b++) {
            int64_t l = S->blist[b];
            for (int64_t e = S->lf_off[l]; e < S->lf_off[l + 1]; e++) {
                int64_t f = S->lf_ids[e];
                if (S->state[f] != ACTIVE || S->frozen_at[f] == sid) continue;
                S->frozen_at[f] = sid;
                S->rate[f] = sstar;
                unfrozen -= 1;
                nnz_u -= S->poff[f + 1] - S->poff[f];
                for (int64_t e2 = S->poff[f]; e2 < S->poff[f + 1]; e2++) {
                    int64_t m = S->plink[e2];
                    if (S->k[m] == 0) S->klist[nk++] = m;
                    S->k[m] += 1;
                }
            }
        }
        /* R_l -= k_l * s*, n_l -= k_l, new share for links still in use */
        for (int64_t q = 0; q < nk; q++) {
            int64_t m = S->klist[q];
            double dec = (double)S->k[m] * sstar;
            S->R[m] = S->R[m] - dec;
            S->n[m] -= S->k[m];
            S->k[m] = 0;
            S->ver[m] += 1;
            if (S->n[m] > 0) {
                if (heap_push(&S->lheap, S->R[m] / (double)S->n[m], m, S->ver[m])) return OR_NOMEM;
            }
        }
        for (int64_t b = 0; b < nb; b++)
            if (S->n[S->blist[b]] != 0) return OR_INTERNAL;
    }
    return OR_OK;
}

typedef struct { double key; int64_t id; } pitem;
typedef struct { pitem* a; int64_t n, cap; } pheap;

static int pheap_push(pheap* h, double key, int64_t id) {
    if (h->n == h->cap) {
        int64_t nc = h->cap ? 2 * h->cap : 1024;
        pitem* na = (pitem*)realloc(h->a, (size_t)nc * sizeof(pitem));
        if (!na) return OR_NOMEM;
        h->a = na; h->cap = nc;
    }
    int64_t i = h->n++;
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (h->a[p].key <= key) break;
        h->a[i] = h->a[p];
        i = p;
    }
    h->a[i].key = key; h->a[i].id = id;
    return OR_OK;
}

static pitem pheap_pop(pheap* h) {
    pitem top = h->a[0];
    pitem last = h->a[--h->n];
    int64_t i = 0;
    for (;;) {
        int64_t c = 2 * i + 1;
        if (c >= h->n) break;
        if (c + 1 < h->n && h->a[c + 1].key < h->a[c].key) c++;
        if (last.key <= h->a[c].key) break;
        h->a[i] = h->a[c];
        i = c;
    }
    if (h->n > 0) h->a[i] = last;
    return top;
}

/*
 * Runs one scenario.  Inputs are validated (see the checks below).
 * counts[0..5) = events, solves, iterations, flows swept, incidences swept,
 * where "swept" sums, over iterations, the unfrozen flows (incidences)
 * present at the start of the iteration.
 * Events later than `until` are not processed (the run stops there and
 * returns 1; flows not finished by then keep finish = NaN).
 * If snap_solve >= 1, the rates right after that solve are copied into
 * snap_rates[F] (0 for flows not active) and its time into *snap_time.
 */
int oracle_run(int64_t L, const double* cap, int64_t F, const double* nbytes,
               const double* start, const double* lat, const int64_t* poff, const int32_t* plink,
               const int64_t* doff, const int64_t* dids, int64_t max_events,
               double until, int64_t snap_solve, double* snap_rates, double* snap_time,
               double* finish, int64_t* counts) {
    for (int i = 0; i < 5; i++) counts[i] = 0;
    if (L < 0 || F < 0) return OR_INVALID;
    for (int64_t l = 0; l < L; l++)
        if (!(cap[l] > 0.0) || !isfinite(cap[l])) return OR_INVALID;
    for (int64_t f = 0; f < F; f++) {
        if (!(nbytes[f] >= 0.0) || !isfinite(nbytes[f])) return OR_INVALID;
        if (!(start[f] >= 0.0) || !isfinite(start[f])) return OR_INVALID;
        if (lat && (!(lat[f] >= 0.0) || !isfinite(lat[f]))) return OR_INVALID;
        if (nbytes[f] > 0.0 && poff[f + 1] == poff[f]) return OR_INVALID;
        for (int64_t e = poff[f]; e < poff[f + 1]; e++)
            if (plink[e] < 0 || plink[e] >= L) return OR_INVALID;
        for (int64_t e = doff[f]; e < doff[f + 1]; e++)
            if (dids[e] < 0 || dids[e] >= f) return OR_INVALID;
    }
    int rc = OR_NOMEM;
    solver S;
    memset(&S, 0, sizeof S);
    S.L = L; S.F = F; S.cap = cap; S.poff = poff; S.plink = plink;
    int64_t nnz = poff[F];
    int64_t nd = doff[F];
    S.lf_off = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.lf_ids = (int64_t*)malloc(((size_t)nnz + 1) * sizeof(int64_t));
    S.R = (double*)malloc(((size_t)L + 1) * sizeof(double));
    S.n = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.k = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.ver = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.stamp = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.touched = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.klist = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.blist = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.state = (uint8_t*)calloc((size_t)F + 1, 1);
    S.frozen_at = (int64_t*)calloc((size_t)F + 1, sizeof(int64_t));
    S.rate = (double*)calloc((size_t)F + 1, sizeof(double));
    double* rem = (double*)calloc((size_t)F + 1, sizeof(double));
    double* tau = (double*)calloc((size_t)F + 1, sizeof(double));
    double* rel_base = (double*)calloc((size_t)F + 1, sizeof(double));
    int64_t* cnt = (int64_t*)calloc((size_t)F + 1, sizeof(int64_t));
    int64_t* s_off = (int64_t*)calloc((size_t)F + 1, sizeof(int64_t));
    int64_t* s_ids = (int64_t*)malloc(((size_t)nd + 1) * sizeof(int64_t));
    int64_t* act = (int64_t*)malloc(((size_t)F + 1) * sizeof(int64_t));
    int64_t* queue = (int64_t*)malloc(((size_t)F + 1) * sizeof(int64_t));
    pheap pend = {0, 0, 0};
    if (!S.lf_off || !S.lf_ids || !S.R || !S.n || !S.k || !S.ver || !S.stamp || !S.touched ||
        !S.klist || !S.blist || !S.state || !S.frozen_at || !S.rate || !rem || !tau ||
        !rel_base || !cnt || !s_off || !s_ids || !act || !queue)
        goto out;

    /* link -> flow transpose */
    for (int64_t e = 0; e < nnz; e++) S.lf_off[plink[e] + 1]++;
    for (int64_t l = 0; l < L; l++) S.lf_off[l + 1] += S.lf_off[l];
    {
        int64_t* fill = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
        if (!fill) goto out;
        memcpy(fill, S.lf_off, (size_t)L * sizeof(int64_t));
        for (int64_t f = 0; f < F; f++)
            for (int64_t e = poff[f]; e < poff[f + 1]; e++) S.lf_ids[fill[plink[e]]++] = f;
        free(fill);
    }
    /* duplicate link inside one path is invalid */
    for (int64_t f = 0; f < F; f++)
        for (int64_t e = poff[f]; e < poff[f + 1]; e++)
            for (int64_t e2 = poff[f]; e2 < e; e2++)
                if (plink[e2] == plink[e]) { rc = OR_INVALID; goto out; }
    /* successor lists from the predecessor lists */
    for (int64_t e = 0; e < nd; e++) s_off[dids[e] + 1]++;
    for (int64_t f = 0; f < F; f++) s_off[f + 1] += s_off[f];
    {
        int64_t* fill = (int64_t*)malloc(((size_t)F + 1) * sizeof(int64_t));
        if (!fill) goto out;
        memcpy(fill, s_off, (size_t)F * sizeof(int64_t));
        for (int64_t g = 0; g < F; g++)
            for (int64_t e = doff[g]; e < doff[g + 1]; e++) s_ids[fill[dids[e]]++] = g;
        free(fill);
    }
    for (int64_t f = 0; f < F; f++) {
        finish[f] = NAN;
        cnt[f] = doff[f + 1] - doff[f];
        if (cnt[f] == 0) {
            S.state[f] = PENDING;
            if (pheap_push(&pend, start[f], f)) goto out;
        } else {
            S.state[f] = WAITING;
        }
    }

    {
        double t = 0.0;
        int64_t na = 0;
        int64_t events = 0, solves = 0;
        for (;;) {
            if (na == 0 && pend.n == 0) break;
            if (max_events > 0 && events >= max_events) { rc = OR_LIMIT; goto out_counts; }
            double t_arr = pend.n ? pend.a[0].key : INFINITY;
            double t_done = INFINITY;
            for (int64_t q = 0; q < na; q++) {
                int64_t f = act[q];
                double dt = rem[f] / S.rate[f];
                tau[f] = t + dt;
                if (tau[f] < t_done) t_done = tau[f];
            }
            double t_next = t_arr < t_done ? t_arr : t_done;
            if (t_next > until) { rc = 1; goto out_counts; }
            events += 1;
            const double thr = t_next * THR;
            const double step = t_next - t;
            int64_t nq = 0, keep = 0;
            for (int64_t q = 0; q < na; q++) {
                int64_t f = act[q];
                if (tau[f] <= thr) {
                    /* the last byte leaves at t_next; it arrives lat[f] later */
                    finish[f] = lat ? t_next + lat[f] : t_next;
                    S.state[f] = DONE;
                    queue[nq++] = f;
                } else {
                    double moved = S.rate[f] * step;
                    rem[f] = rem[f] - moved;
                    act[keep++] = f;
                }
            }
            int changed = nq > 0;
            na = keep;
            t = t_next;
            int64_t qh = 0;
            for (;;) {
                /* release successors of finished flows */
                while (qh < nq) {
                    int64_t f = queue[qh++];
                    for (int64_t e = s_off[f]; e < s_off[f + 1]; e++) {
                        int64_t g = s_ids[e];
                        if (finish[f] > rel_base[g]) rel_base[g] = finish[f];
                        if (--cnt[g] == 0) {
                            S.state[g] = PENDING;
                            if (pheap_push(&pend, start[g] + rel_base[g], g)) goto out;
                        }
                    }
                }
                /* arrivals at or before t */
                int any = 0;
                while (pend.n && pend.a[0].key <= t) {
                    pitem it = pheap_pop(&pend);
                    int64_t g = it.id;
                    if (nbytes[g] == 0.0) {
                        finish[g] = it.key;
                        S.state[g] = DONE;
                        queue[nq++] = g;
                        any = 1;
                    } else {
                        S.state[g] = ACTIVE;
                        rem[g] = nbytes[g];
                        act[na++] = g;
                        changed = 1;
                    }
                }
                if (!any && qh == nq) break;
            }
            if (changed && na > 0) {
                int r = solve(&S, act, na);
                if (r) { rc = r; goto out_counts; }
                solves += 1;
                if (snap_solve == solves && snap_rates) {
                    for (int64_t f = 0; f < F; f++) snap_rates[f] = 0.0;
                    for (int64_t q = 0; q < na; q++) snap_rates[act[q]] = S.rate[act[q]];
                    if (snap_time) *snap_time = t;
                }
            }
            counts[0] = events;
            counts[1] = solves;
        }
        rc = OR_OK;
    }
out_counts:
    counts[2] = S.iterations;
    counts[3] = S.flows_swept;
    counts[4] = S.inc_swept;
out:
    free(S.lf_off); free(S.lf_ids); free(S.R); free(S.n); free(S.k); free(S.ver);
    free(S.stamp); free(S.touched); free(S.klist); free(S.blist); free(S.state);
    free(S.frozen_at); free(S.rate); free(rem); free(tau); free(rel_base); free(cnt);
    free(s_off); free(s_ids); free(act); free(queue); free(S.lheap.a); free(pend.a);
    return rc;
}

/*
 * One rate solve of a given active set (no event loop): rates_out[q] is the
 * rate of flow act[q].  Used to pin the solver on static cases.
 */
int oracle_solve(int64_t L, const double* cap, int64_t F, const int64_t* poff,
                 const int32_t* plink, int64_t na, const int64_t* act, double* rates_out,
                 int64_t* iterations) {
    int rc = OR_NOMEM;
    solver S;
    memset(&S, 0, sizeof S);
    S.L = L; S.F = F; S.cap = cap; S.poff = poff; S.plink = plink;
    int64_t nnz = poff[F];
    for (int64_t l = 0; l < L; l++)
        if (!(cap[l] > 0.0)) return OR_INVALID;
    for (int64_t q = 0; q < na; q++) {
        if (act[q] < 0 || act[q] >= F) return OR_INVALID;
        if (poff[act[q] + 1] == poff[act[q]]) return OR_INVALID;
    }
    S.lf_off = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.lf_ids = (int64_t*)malloc(((size_t)nnz + 1) * sizeof(int64_t));
    S.R = (double*)malloc(((size_t)L + 1) * sizeof(double));
    S.n = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.k = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.ver = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.stamp = (int64_t*)calloc((size_t)L + 1, sizeof(int64_t));
    S.touched = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.klist = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.blist = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
    S.state = (uint8_t*)calloc((size_t)F + 1, 1);
    S.frozen_at = (int64_t*)calloc((size_t)F + 1, sizeof(int64_t));
    S.rate = (double*)calloc((size_t)F + 1, sizeof(double));
    if (!S.lf_off || !S.lf_ids || !S.R || !S.n || !S.k || !S.ver || !S.stamp || !S.touched ||
        !S.klist || !S.blist || !S.state || !S.frozen_at || !S.rate)
        goto out;
    for (int64_t e = 0; e < nnz; e++) S.lf_off[plink[e] + 1]++;
    for (int64_t l = 0; l < L; l++) S.lf_off[l + 1] += S.lf_off[l];
    {
        int64_t* fill = (int64_t*)malloc(((size_t)L + 1) * sizeof(int64_t));
        if (!fill) goto out;
        memcpy(fill, S.lf_off, (size_t)L * sizeof(int64_t));
        for (int64_t f = 0; f < F; f++)
            for (int64_t e = poff[f]; e < poff[f + 1]; e++) S.lf_ids[fill[plink[e]]++] = f;
        free(fill);
    }
    for (int64_t q = 0; q < na; q++) S.state[act[q]] = ACTIVE;
    rc = na > 0 ? solve(&S, act, na) : OR_OK;
    if (rc == OR_OK)
        for (int64_t q = 0; q < na; q++) rates_out[q] = S.rate[act[q]];
    if (iterations) *iterations = S.iterations;
out:
    free(S.lf_off); free(S.lf_ids); free(S.R); free(S.n); free(S.k); free(S.ver);
    free(S.stamp); free(S.touched); free(S.klist); free(S.blist); free(S.state);
    free(S.frozen_at); free(S.rate); free(S.lheap.a);
    return rc;
}

/*
 * dd_oracle.c -- TEST INFRASTRUCTURE ONLY (the oracle).
 *
 * A plain, slow CPU reference for the batched what-if simulation.  For each
 * requested variant it
 *   1. applies the graph transformations of Sec. 4.4: the shrink/scale
 *      primitive (duration * p / q, floored to whole nanoseconds) and the
 *      Remove primitive; edges whose class is switched off in the variant
 *      are absent;
 *   2. runs the simulation of Sec. 4.1, Algorithm 1, step by step: reference
 *      counts over every task's parents, a frontier F of ready tasks,
 *      schedule(F) picking the task with the earliest start (Sec. 4.4,
 *      "Schedule"), per-thread progress P[t], start = max(P[t], start),
 *      P[t] = start + duration + gap, and every child's start raised to the
 *      parent's start + duration + gap.
 * Parents are the dependency edges of Sec. 4.2.2 given in the input plus
 * the order of consecutive tasks on one execution thread (also a dependency
 * type of Sec. 4.2.2).
 *
 * A third entry point runs the same loop with an overridden schedule()
 * (Sec. 4.4, "Schedule"; the appendix's P3 priority rule) on graphs whose
 * threads may hold tasks with no order among them.
 *
 * Removal has two readings, both implemented so tests can check that they
 * agree: mode 0 keeps a removed task with duration and gap 0 (a
 * pass-through); mode 1 unlinks it (Sec. 4.4, Insert/Remove: the task is
 * taken out of its thread's list, and each of its predecessors is linked to
 * each of its successors).
 *
 * Only tests/, the smoke check and the CPU-baseline leg of the benchmark may
 * load this library.  It shares no code, header or table with the GPU path.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n;
    int32_t n_threads;
    const int64_t *in_ptr;     /* [n+1] */
    const int32_t *in_src;     /* [E]   */
    const uint8_t *edge_cls;   /* [E]   */
    const int32_t *thread_prev;/* [n]   */
    const int32_t *thread_id;  /* [n]   */
    const int64_t *dur;        /* [n]   */
    const int64_t *gap;        /* [n]   */
    const uint16_t *node_cls;  /* [n]   */
} ddo_graph;

typedef struct {
    int32_t n_variants;        /* V: columns of the tables */
    int32_t n_cls;
    const int32_t *scale;      /* [n_cls][V][2] (p, q) */
    const uint32_t *rm_bits;   /* [n][ceil(V/32)] */
    int32_t edge_words;
    const uint64_t *edge_on;   /* [V][edge_words] */
} ddo_variants;

enum { DDO_OK = 0, DDO_EINVAL = 1, DDO_ECYCLE = 2, DDO_ENOMEM = 5 };

/* ------------------------------------------------------------------ */
/* shared, variant-independent structure: out-edges (children) */
typedef struct {
    int64_t *out_ptr;  /* [n+1] */
    int32_t *out_dst;  /* [E]   */
    uint8_t *out_cls;  /* [E]   */
    int32_t *thread_next; /* [n] */
} ddo_struct;

static int build_struct(const ddo_graph *g, ddo_struct *s) {
    int32_t n = g->n;
    int64_t E = g->in_ptr[n];
    s->out_ptr = calloc((size_t)n + 1, sizeof(int64_t));
    s->out_dst = malloc((size_t)(E > 0 ? E : 1) * sizeof(int32_t));
    s->out_cls = malloc((size_t)(E > 0 ? E : 1));
    s->thread_next = malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!s->out_ptr || !s->out_dst || !s->out_cls || !s->thread_next) return DDO_ENOMEM;
    for (int32_t v = 0; v < n; v++)
        for (int64_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) s->out_ptr[g->in_src[e] + 1]++;
    for (int32_t u = 0; u < n; u++) s->out_ptr[u + 1] += s->out_ptr[u];
    int64_t *fill = malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!fill) return DDO_ENOMEM;
    for (int32_t u = 0; u < n; u++) fill[u] = s->out_ptr[u];
    for (int32_t v = 0; v < n; v++)
        for (int64_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) {
            int32_t u = g->in_src[e];
            s->out_dst[fill[u]] = v;
            s->out_cls[fill[u]] = g->edge_cls ? g->edge_cls[e] : 0;
            fill[u]++;
        }
    free(fill);
    for (int32_t u = 0; u < n; u++) s->thread_next[u] = -1;
    for (int32_t u = 0; u < n; u++)
        if (g->thread_prev[u] >= 0) s->thread_next[g->thread_prev[u]] = u;
    return DDO_OK;
}

static void free_struct(ddo_struct *s) {
    free(s->out_ptr); free(s->out_dst); free(s->out_cls); free(s->thread_next);
}

/* ------------------------------------------------------------------ */
/* frontier: binary min-heap ordered by (start, tie key, id) */
typedef struct { int64_t key; int64_t tie; int32_t id; } hnode;
typedef struct { hnode *a; int32_t n; } heap;

static int hless(const hnode *x, const hnode *y) {
    if (x->key != y->key) return x->key < y->key;
    if (x->tie != y->tie) return x->tie < y->tie;
    return x->id < y->id;
}
static void hpush(heap *h, hnode x) {
    int32_t i = h->n++;
    h->a[i] = x;
    while (i > 0) {
        int32_t p = (i - 1) / 2;
        if (!hless(&h->a[i], &h->a[p])) break;
        hnode t = h->a[i]; h->a[i] = h->a[p]; h->a[p] = t; i = p;
    }
}
static hnode hpop(heap *h) {
    hnode top = h->a[0];
    h->a[0] = h->a[--h->n];
    int32_t i = 0;
    for (;;) {
        int32_t l = 2 * i + 1, r = l + 1, m = i;
        if (l < h->n && hless(&h->a[l], &h->a[m])) m = l;
        if (r < h->n && hless(&h->a[r], &h->a[m])) m = r;
        if (m == i) break;
        hnode t = h->a[i]; h->a[i] = h->a[m]; h->a[m] = t; i = m;
    }
    return top;
}

/* tie rule of schedule() among tasks with the same start:
 * 0 = earliest in the trace (lowest id), 1 = latest in the trace,
 * 2 = lowest execution thread, then lowest id. */
static int64_t tie_key(const ddo_graph *g, int32_t u, int tie) {
    if (tie == 1) return -(int64_t)u;
    if (tie == 2) return (int64_t)g->thread_id[u];
    return (int64_t)u;
}

/* ------------------------------------------------------------------ */
static int is_removed(const ddo_variants *vs, int32_t u, int32_t v) {
    if (!vs->rm_bits) return 0;
    int32_t W = (vs->n_variants + 31) / 32;
    return (int)((vs->rm_bits[(int64_t)u * W + v / 32] >> (v % 32)) & 1u);
}
static int edge_active(const ddo_variants *vs, int32_t v, int cls) {
    if (!vs->edge_on) return 1;
    uint64_t w = vs->edge_on[(int64_t)v * vs->edge_words + cls / 64];
    return (int)((w >> (cls % 64)) & 1u);
}

/* shrink/scale: floor(d * p / q) in exact integer arithmetic */
static int64_t scaled(int64_t d, int32_t p, int32_t q) {
    __int128 a = (__int128)d * (__int128)p;
    return (int64_t)(a / (__int128)q);
}

typedef struct {
    int64_t *dd, *gg, *est, *S;     /* per task */
    int32_t *ref;
    uint8_t *rm, *done;
    int64_t *P;                     /* per thread */
    hnode *heapbuf;
    /* unlink mode: effective parents */
    int64_t *ep_ptr; int32_t *ep; int64_t ep_cap;
    int32_t *ep_cnt;
} work;

/* Mode 1 helper: push the parents of task x present in variant v. */
static void push_parents(const ddo_graph *g, const ddo_variants *vs, int32_t v, int32_t x,
                         uint8_t *seen, int32_t *stack, int64_t *sp,
                         int32_t *touched, int64_t *ntouched) {
    for (int64_t e = g->in_ptr[x]; e < g->in_ptr[x + 1]; e++) {
        int c = g->edge_cls ? g->edge_cls[e] : 0;
        if (!edge_active(vs, v, c)) continue;
        int32_t q = g->in_src[e];
        if (!seen[q]) { seen[q] = 1; touched[(*ntouched)++] = q; stack[(*sp)++] = q; }
    }
    int32_t q = g->thread_prev[x];
    if (q >= 0 && !seen[q]) { seen[q] = 1; touched[(*ntouched)++] = q; stack[(*sp)++] = q; }
}

/* Mode 1 helper: the kept tasks that the parents of u lead back to when
 * removed tasks are contracted away. */
static int collect_eff(const ddo_graph *g, const ddo_variants *vs, int32_t v, int32_t u,
                       int32_t **outp, int64_t *outn, int64_t *outcap, uint8_t *seen,
                       int32_t *stack, int32_t *touched, int64_t *ntouched) {
    int64_t sp = 0;
    push_parents(g, vs, v, u, seen, stack, &sp, touched, ntouched);
    while (sp > 0) {
        int32_t p = stack[--sp];
        if (is_removed(vs, p, v)) {
            push_parents(g, vs, v, p, seen, stack, &sp, touched, ntouched);
        } else {
            if (*outn >= *outcap) {
                *outcap = *outcap * 2 + 16;
                int32_t *np_ = realloc(*outp, (size_t)*outcap * sizeof(int32_t));
                if (!np_) return DDO_ENOMEM;
                *outp = np_;
            }
            (*outp)[(*outn)++] = p;
        }
    }
    return DDO_OK;
}

static int run_variant(const ddo_graph *g, const ddo_struct *st, const ddo_variants *vs,
                       int32_t v, int mode, int tie, work *w,
                       int64_t *start_row, int64_t *finish_row, int64_t *makespan,
                       int64_t *bindings) {
    const int32_t n = g->n;
    int32_t V = vs->n_variants;
    /* 1. transformations */
    for (int32_t u = 0; u < n; u++) {
        int r = is_removed(vs, u, v);
        w->rm[u] = (uint8_t)r;
        int32_t p = 1, q = 1;
        if (vs->scale) {
            int64_t o = ((int64_t)g->node_cls[u] * V + v) * 2;
            p = vs->scale[o];
            q = vs->scale[o + 1];
        }
        w->dd[u] = r ? 0 : scaled(g->dur[u], p, q);
        w->gg[u] = r ? 0 : g->gap[u];
    }
    int64_t nb = 0;
    heap h = { w->heapbuf, 0 };
    for (int32_t t = 0; t < g->n_threads; t++) w->P[t] = 0;   /* P <- {0} */

    if (mode == 0) {
        /* 2. reference counts over all parents (lines: ref <- |parents|) */
        for (int32_t u = 0; u < n; u++) {
            int32_t r = (g->thread_prev[u] >= 0) ? 1 : 0;
            for (int64_t e = g->in_ptr[u]; e < g->in_ptr[u + 1]; e++) {
                int c = g->edge_cls ? g->edge_cls[e] : 0;
                if (edge_active(vs, v, c)) r++;
            }
            w->ref[u] = r;
            w->est[u] = 0;
            w->done[u] = 0;
        }
        for (int32_t u = 0; u < n; u++)
            if (w->ref[u] == 0) {
                hnode x = { 0, tie_key(g, u, tie), u };
                hpush(&h, x);
            }
        int32_t dispatched = 0;
        while (h.n > 0) {
            hnode x = hpop(&h);                       /* u <- schedule(F) */
            int32_t u = x.id;
            int32_t t = g->thread_id[u];              /* t <- u.ExecutionThread */
            if (w->P[t] > w->est[u]) nb++;
            int64_t s = w->P[t] > w->est[u] ? w->P[t] : w->est[u];   /* u.start */
            w->S[u] = s;
            int64_t rel = s + w->dd[u] + w->gg[u];
            w->P[t] = rel;                            /* thread progress */
            w->done[u] = 1;
            dispatched++;
            /* children: dependency out-edges and the next task on the thread */
            for (int64_t e = st->out_ptr[u]; e < st->out_ptr[u + 1]; e++) {
                if (!edge_active(vs, v, st->out_cls[e])) continue;
                int32_t c = st->out_dst[e];
                if (rel > w->est[c]) w->est[c] = rel;
                if (--w->ref[c] == 0) {
                    int32_t tc = g->thread_id[c];
                    int64_t k = w->P[tc] > w->est[c] ? w->P[tc] : w->est[c];
                    hnode y = { k, tie_key(g, c, tie), c };
                    hpush(&h, y);
                }
            }
            int32_t c = st->thread_next[u];
            if (c >= 0) {
                if (rel > w->est[c]) w->est[c] = rel;
                if (--w->ref[c] == 0) {
                    int32_t tc = g->thread_id[c];
                    int64_t k = w->P[tc] > w->est[c] ? w->P[tc] : w->est[c];
                    hnode y = { k, tie_key(g, c, tie), c };
                    hpush(&h, y);
                }
            }
        }
        if (dispatched != n) return DDO_ECYCLE;
    } else {
        /* unlink mode: effective parents of every task through removed ones */
        uint8_t *seen = calloc((size_t)n + 1, 1);
        int32_t *stack = malloc(((size_t)n + 1) * sizeof(int32_t) * 2);
        int32_t *touched = malloc(((size_t)n + 1) * sizeof(int32_t));
        int64_t *eptr = malloc(((size_t)n + 1) * sizeof(int64_t));
        int32_t *eps = NULL; int64_t nep = 0, cap = 0;
        if (!seen || !stack || !touched || !eptr) return DDO_ENOMEM;
        for (int32_t u = 0; u < n; u++) {
            eptr[u] = nep;
            int64_t nt = 0;
            int rc = collect_eff(g, vs, v, u, &eps, &nep, &cap, seen, stack, touched, &nt);
            if (rc) return rc;
            for (int64_t i = 0; i < nt; i++) seen[touched[i]] = 0;
        }
        eptr[n] = nep;
        /* children lists from effective parents (kept tasks only) */
        int64_t *cptr = calloc((size_t)n + 1, sizeof(int64_t));
        int32_t *cs = malloc((size_t)(nep > 0 ? nep : 1) * sizeof(int32_t));
        if (!cptr || !cs) return DDO_ENOMEM;
        for (int32_t u = 0; u < n; u++)
            if (!w->rm[u])
                for (int64_t i = eptr[u]; i < eptr[u + 1]; i++) cptr[eps[i] + 1]++;
        for (int32_t u = 0; u < n; u++) cptr[u + 1] += cptr[u];
        int64_t *fill = malloc(((size_t)n + 1) * sizeof(int64_t));
        for (int32_t u = 0; u <= n; u++) fill[u] = cptr[u];
        for (int32_t u = 0; u < n; u++)
            if (!w->rm[u])
                for (int64_t i = eptr[u]; i < eptr[u + 1]; i++) cs[fill[eps[i]]++] = u;
        int32_t kept = 0;
        for (int32_t u = 0; u < n; u++) {
            w->est[u] = 0;
            w->ref[u] = (int32_t)(eptr[u + 1] - eptr[u]);
            w->done[u] = 0;
            if (!w->rm[u]) kept++;
        }
        for (int32_t u = 0; u < n; u++)
            if (!w->rm[u] && w->ref[u] == 0) {
                hnode x = { 0, tie_key(g, u, tie), u };
                hpush(&h, x);
            }
        int32_t dispatched = 0;
        while (h.n > 0) {
            hnode x = hpop(&h);
            int32_t u = x.id;
            int32_t t = g->thread_id[u];
            if (w->P[t] > w->est[u]) nb++;
            int64_t s = w->P[t] > w->est[u] ? w->P[t] : w->est[u];
            w->S[u] = s;
            int64_t rel = s + w->dd[u] + w->gg[u];
            w->P[t] = rel;
            w->done[u] = 1;
            dispatched++;
            for (int64_t i = cptr[u]; i < cptr[u + 1]; i++) {
                int32_t c = cs[i];
                if (rel > w->est[c]) w->est[c] = rel;
                if (--w->ref[c] == 0) {
                    int32_t tc = g->thread_id[c];
                    int64_t k = w->P[tc] > w->est[c] ? w->P[tc] : w->est[c];
                    hnode y = { k, tie_key(g, c, tie), c };
                    hpush(&h, y);
                }
            }
        }
        int rc = (dispatched != kept) ? DDO_ECYCLE : DDO_OK;
        /* a removed task reports the moment its inputs are all available */
        if (rc == DDO_OK)
            for (int32_t u = 0; u < n; u++)
                if (w->rm[u]) {
                    int64_t s = 0;
                    for (int64_t i = eptr[u]; i < eptr[u + 1]; i++) {
                        int32_t p = eps[i];
                        int64_t r = w->S[p] + w->dd[p] + w->gg[p];
                        if (r > s) s = r;
                    }
                    w->S[u] = s;
                }
        free(seen); free(stack); free(touched); free(eptr); free(eps);
        free(cptr); free(cs); free(fill);
        if (rc) return rc;
    }
    /* outputs: start, finish = start + duration, makespan over kept tasks */
    int64_t ms = 0;
    for (int32_t u = 0; u < n; u++) {
        int64_t f = w->S[u] + w->dd[u];
        if (start_row) start_row[u] = w->S[u];
        if (finish_row) finish_row[u] = f;
        if (!w->rm[u] && f > ms) ms = f;
    }
    *makespan = ms;
    if (bindings) *bindings = nb;
    return DDO_OK;
}

/* ------------------------------------------------------------------ */
/* The simulation under an overridden schedule() (Sec. 4.4, "Schedule"; the
 * appendix's P3 model).  Same transformations and the same loop as above
 * (removed tasks kept with zero duration and gap), but threads may hold
 * tasks with no order among them (several chains on one thread, e.g. the
 * push and pull slices on a communication channel), so which ready task runs
 * next decides the result.  The frontier Q is kept in trace order (ascending
 * task id); Q.first() is its lowest id.  schedule(Q) scans Q in that order
 * with time(x) = max(P[x.thread], x.start):
 *   policy 0 (the default rule): the first task of least time;
 *   policy 1 (P3's priority rule): the same scan, where a later task of equal
 *            time also replaces the current choice when both are push/pull
 *            tasks (pp[] != 0) and its priority is strictly higher.
 * A task is dispatched at max(P[t], start); its thread's progress becomes its
 * start + duration + gap, and so does every child's start if larger. */
static int run_variant_policy(const ddo_graph *g, const ddo_struct *st, const ddo_variants *vs,
                              int32_t v, int policy, const uint8_t *pp, const int32_t *prio,
                              work *w, int64_t *start_row, int64_t *finish_row,
                              int64_t *makespan) {
    const int32_t n = g->n;
    const int32_t V = vs->n_variants;
    int32_t *Q = (int32_t *)w->heapbuf;
    int32_t qn = 0;
    for (int32_t u = 0; u < n; u++) {
        int r = is_removed(vs, u, v);
        w->rm[u] = (uint8_t)r;
        int32_t p = 1, q = 1;
        if (vs->scale) {
            int64_t o = ((int64_t)g->node_cls[u] * V + v) * 2;
            p = vs->scale[o];
            q = vs->scale[o + 1];
        }
        w->dd[u] = r ? 0 : scaled(g->dur[u], p, q);
        w->gg[u] = r ? 0 : g->gap[u];
    }
    for (int32_t t = 0; t < g->n_threads; t++) w->P[t] = 0;
    for (int32_t u = 0; u < n; u++) {
        int32_t r = (g->thread_prev[u] >= 0) ? 1 : 0;
        for (int64_t e = g->in_ptr[u]; e < g->in_ptr[u + 1]; e++) {
            int c = g->edge_cls ? g->edge_cls[e] : 0;
            if (edge_active(vs, v, c)) r++;
        }
        w->ref[u] = r;
        w->est[u] = 0;
        if (r == 0) Q[qn++] = u;                       /* ids ascending */
    }
    int32_t dispatched = 0;
    while (qn > 0) {
        /* u <- schedule(Q) */
        int32_t bi = 0;
        int32_t best = Q[0];
        int64_t time = w->P[g->thread_id[best]] > w->est[best] ? w->P[g->thread_id[best]]
                                                             : w->est[best];
        for (int32_t i = 0; i < qn; i++) {
            int32_t x = Q[i];
            int64_t px = w->P[g->thread_id[x]];
            int64_t tx = px > w->est[x] ? px : w->est[x];
            if (tx < time) { time = tx; best = x; bi = i; }
            if (policy == 1 && tx == time && pp[x] && pp[best] && prio[x] > prio[best]) {
                best = x;
                bi = i;
            }
        }
        memmove(&Q[bi], &Q[bi + 1], (size_t)(qn - bi - 1) * sizeof(int32_t));
        qn--;
        int32_t u = best;
        int32_t t = g->thread_id[u];
        int64_t s = w->P[t] > w->est[u] ? w->P[t] : w->est[u];
        w->S[u] = s;
        int64_t rel = s + w->dd[u] + w->gg[u];
        w->P[t] = rel;
        dispatched++;
        /* children: dependency out-edges, then the next task on the thread */
        for (int64_t e = st->out_ptr[u]; e <= st->out_ptr[u + 1]; e++) {
            int32_t c;
            if (e < st->out_ptr[u + 1]) {
                if (!edge_active(vs, v, st->out_cls[e])) continue;
                c = st->out_dst[e];
            } else {
                c = st->thread_next[u];
                if (c < 0) break;
            }
            if (rel > w->est[c]) w->est[c] = rel;
            if (--w->ref[c] == 0) {                    /* insert, keeping Q in id order */
                int32_t i = qn;
                while (i > 0 && Q[i - 1] > c) { Q[i] = Q[i - 1]; i--; }
                Q[i] = c;
                qn++;
            }
        }
    }
    if (dispatched != n) return DDO_ECYCLE;
    int64_t ms = 0;
    for (int32_t u = 0; u < n; u++) {
        int64_t f = w->S[u] + w->dd[u];
        if (start_row) start_row[u] = w->S[u];
        if (finish_row) finish_row[u] = f;
        if (!w->rm[u] && f > ms) ms = f;
    }
    *makespan = ms;
    return DDO_OK;
}

/* ------------------------------------------------------------------ */
/* Runtime breakdown of the evaluation of AMP (Sec. 6.2, Fig. 6), from one
 * variant's simulated schedule, by the paper's own rules for computing it:
 *   total    = the iteration time (makespan);
 *   CPU-only = total minus all GPU kernel runtime (the kernels' durations);
 *   GPU-only = the time the CPU is blocked waiting for the GPU: for every
 *              synchronization call and every device-to-host copy call, from
 *              the moment its thread reached it (the release of the previous
 *              task on the thread, 0 for the first) to the moment it starts
 *              (the simulation starts it when the GPU work it waits on is done;
 *              its own duration is the call's CPU time);
 *   CPU+GPU parallel = total - CPU-only - GPU-only.
 * role[u]: 1 = GPU kernel, 2 = CPU call that waits for the GPU, 0 = other. */
static void breakdown(const ddo_graph *g, const uint8_t *role, const work *w, int64_t ms,
                      int64_t *out) {
    int64_t gpu = 0, wait = 0;
    for (int32_t u = 0; u < g->n; u++) {
        if (role[u] == 1) gpu += w->dd[u];
        if (role[u] == 2) {
            int32_t p = g->thread_prev[u];
            int64_t reached = p >= 0 ? w->S[p] + w->dd[p] + w->gg[p] : 0;
            wait += w->S[u] - reached;
        }
    }
    out[0] = ms;
    out[1] = ms - gpu;
    out[2] = wait;
    out[3] = ms - out[1] - out[2];
}

typedef struct {
    const ddo_graph *g; const ddo_struct *st; const ddo_variants *vs;
    const int32_t *vlist; int32_t n_list; int mode, tie;
    int64_t *start, *finish, *makespan, *bindings;
    const uint8_t *role; int64_t *bd;        /* breakdown: role [n] in, [n_list][4] out */
    int policy; const uint8_t *pp; const int32_t *prio;   /* policy >= 0: run_variant_policy */
    int32_t next; pthread_mutex_t mu; int rc;
} job;

static void *worker(void *arg) {
    job *j = (job *)arg;
    const int32_t n = j->g->n;
    work w;
    memset(&w, 0, sizeof(w));
    size_t nn = (size_t)(n > 0 ? n : 1);
    w.dd = malloc(nn * 8); w.gg = malloc(nn * 8); w.est = malloc(nn * 8); w.S = malloc(nn * 8);
    w.ref = malloc(nn * 4); w.rm = malloc(nn); w.done = malloc(nn);
    w.P = malloc((size_t)(j->g->n_threads > 0 ? j->g->n_threads : 1) * 8);
    w.heapbuf = malloc(nn * sizeof(hnode));
    int ok = w.dd && w.gg && w.est && w.S && w.ref && w.rm && w.done && w.P && w.heapbuf;
    for (;;) {
        pthread_mutex_lock(&j->mu);
        int32_t i = j->next++;
        if (!ok && j->rc == 0) j->rc = DDO_ENOMEM;
        pthread_mutex_unlock(&j->mu);
        if (i >= j->n_list || !ok) break;
        int32_t v = j->vlist[i];
        int rc = j->policy >= 0
            ? run_variant_policy(j->g, j->st, j->vs, v, j->policy, j->pp, j->prio, &w,
                                 j->start ? j->start + (int64_t)i * n : NULL,
                                 j->finish ? j->finish + (int64_t)i * n : NULL,
                                 &j->makespan[i])
            : run_variant(j->g, j->st, j->vs, v, j->mode, j->tie, &w,
                          j->start ? j->start + (int64_t)i * n : NULL,
                          j->finish ? j->finish + (int64_t)i * n : NULL,
                          &j->makespan[i], j->bindings ? &j->bindings[i] : NULL);
        if (rc) {
            pthread_mutex_lock(&j->mu);
            if (j->rc == 0) j->rc = rc;
            pthread_mutex_unlock(&j->mu);
        } else if (j->role) {
            breakdown(j->g, j->role, &w, j->makespan[i], j->bd + (int64_t)i * 4);
        }
    }
    free(w.dd); free(w.gg); free(w.est); free(w.S); free(w.ref); free(w.rm); free(w.done);
    free(w.P); free(w.heapbuf);
    return NULL;
}

/* Basic argument checks; the oracle trusts the structure otherwise except for
 * cycles, which it reports as DDO_ECYCLE. */
static int check(const ddo_graph *g, const ddo_variants *vs) {
    if (g->n < 0 || g->n_threads < 0) return DDO_EINVAL;
    for (int32_t u = 0; u < g->n; u++) {
        if (g->thread_id[u] < 0 || g->thread_id[u] >= g->n_threads) return DDO_EINVAL;
        if (g->dur[u] < 0 || g->gap[u] < 0) return DDO_EINVAL;
        int32_t p = g->thread_prev[u];
        if (p < -1 || p >= g->n) return DDO_EINVAL;
        if (vs->scale && g->node_cls[u] >= vs->n_cls) return DDO_EINVAL;
    }
    for (int64_t e = 0; e < g->in_ptr[g->n]; e++)
        if (g->in_src[e] < 0 || g->in_src[e] >= g->n) return DDO_EINVAL;
    if (vs->scale)
        for (int64_t i = 0; i < (int64_t)vs->n_cls * vs->n_variants; i++)
            if (vs->scale[2 * i] < 0 || vs->scale[2 * i + 1] < 1) return DDO_EINVAL;
    return DDO_OK;
}

static int run_job(const ddo_graph *g, const ddo_variants *vs,
                   const int32_t *vlist, int32_t n_list, int32_t mode, int32_t tie,
                   int64_t *start, int64_t *finish, int64_t *makespan, int64_t *bindings,
                   const uint8_t *role, int64_t *bd, int32_t n_workers,
                   int policy, const uint8_t *pp, const int32_t *prio);

int ddo_run(const ddo_graph *g, const ddo_variants *vs,
            const int32_t *vlist, int32_t n_list, int32_t mode, int32_t tie,
            int64_t *start, int64_t *finish, int64_t *makespan, int64_t *bindings,
            int32_t n_workers) {
    return run_job(g, vs, vlist, n_list, mode, tie, start, finish, makespan, bindings, NULL, NULL,
                   n_workers, -1, NULL, NULL);
}

/* The simulation of each listed variant under schedule policy 0 or 1 (see
 * run_variant_policy); pp and prio [n] are read by policy 1 only. */
int ddo_run_policy(const ddo_graph *g, const ddo_variants *vs, const int32_t *vlist,
                   int32_t n_list, int32_t policy, const uint8_t *pp, const int32_t *prio,
                   int64_t *start, int64_t *finish, int64_t *makespan, int32_t n_workers) {
    if (policy != 0 && policy != 1) return DDO_EINVAL;
    if (policy == 1 && (!pp || !prio)) return DDO_EINVAL;
    return run_job(g, vs, vlist, n_list, 0, 0, start, finish, makespan, NULL, NULL, NULL,
                   n_workers, policy, pp, prio);
}

/* The runtime breakdown (see breakdown()) of each listed variant after the
 * simulation (mode 0): out [n_list][4] = total, CPU-only, GPU-only,
 * CPU+GPU parallel. */
int ddo_breakdown(const ddo_graph *g, const ddo_variants *vs, const uint8_t *role,
                  const int32_t *vlist, int32_t n_list, int64_t *makespan, int64_t *out,
                  int32_t n_workers) {
    if (!role) return DDO_EINVAL;
    return run_job(g, vs, vlist, n_list, 0, 0, NULL, NULL, makespan, NULL, role, out, n_workers,
                   -1, NULL, NULL);
}

static int run_job(const ddo_graph *g, const ddo_variants *vs,
                   const int32_t *vlist, int32_t n_list, int32_t mode, int32_t tie,
                   int64_t *start, int64_t *finish, int64_t *makespan, int64_t *bindings,
                   const uint8_t *role, int64_t *bd, int32_t n_workers,
                   int policy, const uint8_t *pp, const int32_t *prio) {
    int rc = check(g, vs);
    if (rc) return rc;
    for (int32_t i = 0; i < n_list; i++)
        if (vlist[i] < 0 || vlist[i] >= vs->n_variants) return DDO_EINVAL;
    ddo_struct st;
    memset(&st, 0, sizeof(st));
    rc = build_struct(g, &st);
    if (rc) { free_struct(&st); return rc; }
    job j;
    memset(&j, 0, sizeof(j));
    j.g = g; j.st = &st; j.vs = vs; j.vlist = vlist; j.n_list = n_list;
    j.mode = mode; j.tie = tie; j.start = start; j.finish = finish;
    j.makespan = makespan; j.bindings = bindings; j.role = role; j.bd = bd;
    j.policy = policy; j.pp = pp; j.prio = prio;
    pthread_mutex_init(&j.mu, NULL);
    if (n_workers < 1) n_workers = 1;
    if (n_workers > n_list) n_workers = n_list > 0 ? n_list : 1;
    pthread_t *th = malloc(sizeof(pthread_t) * (size_t)n_workers);
    for (int32_t i = 0; i < n_workers; i++) pthread_create(&th[i], NULL, worker, &j);
    for (int32_t i = 0; i < n_workers; i++) pthread_join(th[i], NULL);
    free(th);
    pthread_mutex_destroy(&j.mu);
    free_struct(&st);
    return j.rc;
}

/* ------------------------------------------------------------------ */
/* Topological steps of the graph restricted to the edge classes in `mask`
 * (thread order always present), by Kahn's algorithm (the reference counts
 * and frontier of Sec. 4.1, Algorithm 1, popped first-in first-out):
 *   level[u] = longest path to u counted in edges (Kahn level);
 *   phase[u] = longest path to u where a dependency between two different
 *              threads counts 1 and thread order (or a dependency inside
 *              one thread) counts 0.
 * Returns DDO_ECYCLE if some task is never freed. */
int ddo_steps(const ddo_graph *g, uint64_t mask, int32_t *level, int32_t *phase) {
    const int32_t n = g->n;
    ddo_struct st;
    memset(&st, 0, sizeof(st));
    int rc = build_struct(g, &st);
    int32_t *ref = malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    int32_t *queue = malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (rc || !ref || !queue) { free_struct(&st); free(ref); free(queue); return DDO_ENOMEM; }
    for (int32_t u = 0; u < n; u++) {
        int32_t r = g->thread_prev[u] >= 0 ? 1 : 0;
        for (int64_t e = g->in_ptr[u]; e < g->in_ptr[u + 1]; e++) {
            int c = g->edge_cls ? g->edge_cls[e] : 0;
            if ((mask >> c) & 1u) r++;
        }
        ref[u] = r;
        level[u] = 0;
        phase[u] = 0;
    }
    int32_t head = 0, tail = 0;
    for (int32_t u = 0; u < n; u++)
        if (ref[u] == 0) queue[tail++] = u;
    while (head < tail) {
        int32_t u = queue[head++];
        for (int64_t e = st.out_ptr[u]; e < st.out_ptr[u + 1]; e++) {
            if (!((mask >> st.out_cls[e]) & 1u)) continue;
            int32_t c = st.out_dst[e];
            int32_t w = g->thread_id[c] != g->thread_id[u] ? 1 : 0;
            if (level[u] + 1 > level[c]) level[c] = level[u] + 1;
            if (phase[u] + w > phase[c]) phase[c] = phase[u] + w;
            if (--ref[c] == 0) queue[tail++] = c;
        }
        int32_t c = st.thread_next[u];
        if (c >= 0) {
            if (level[u] + 1 > level[c]) level[c] = level[u] + 1;
            if (phase[u] > phase[c]) phase[c] = phase[u];
            if (--ref[c] == 0) queue[tail++] = c;
        }
    }
    free_struct(&st);
    free(ref);
    free(queue);
    return tail == n ? DDO_OK : DDO_ECYCLE;
}

/* Runs the oracle under AddressSanitizer and UBSan on one input file and
 * writes its outputs, so the test can compare them with the normal build.
 * Input (little endian): int32 n, n_threads, V, n_cls, edge_words;
 * int64 E; then in_ptr[n+1] i64, in_src[E] i32, edge_cls[E] u8,
 * thread_prev[n] i32, thread_id[n] i32, dur[n] i64, gap[n] i64,
 * node_cls[n] u16, scale[n_cls*V*2] i32, rm_bits[n*ceil(V/32)] u32,
 * edge_on[V*edge_words] u64.
 * Output: for mode 0 and 1, ties 0..2, workers 1 and 3: start, finish,
 * makespan of every variant (i64); then Kahn level and phase (i32). */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n, n_threads;
    const int64_t *in_ptr; const int32_t *in_src; const uint8_t *edge_cls;
    const int32_t *thread_prev; const int32_t *thread_id;
    const int64_t *dur; const int64_t *gap; const uint16_t *node_cls;
} ddo_graph;
typedef struct {
    int32_t n_variants, n_cls;
    const int32_t *scale; const uint32_t *rm_bits;
    int32_t edge_words; const uint64_t *edge_on;
} ddo_variants;
int ddo_run(const ddo_graph *, const ddo_variants *, const int32_t *, int32_t, int32_t, int32_t,
            int64_t *, int64_t *, int64_t *, int64_t *, int32_t);
int ddo_steps(const ddo_graph *, uint64_t, int32_t *, int32_t *);

static void *rd(FILE *f, size_t bytes) {
    void *p = malloc(bytes ? bytes : 1);
    if (bytes && fread(p, 1, bytes, f) != bytes) { fprintf(stderr, "short read\n"); exit(2); }
    return p;
}

int main(int argc, char **argv) {
    if (argc != 3) return 2;
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t h[5];
    int64_t E;
    if (fread(h, 4, 5, f) != 5 || fread(&E, 8, 1, f) != 1) return 2;
    int32_t n = h[0], T = h[1], V = h[2], C = h[3], K = h[4];
    int32_t W = (V + 31) / 32;
    ddo_graph g;
    g.n = n; g.n_threads = T;
    g.in_ptr = rd(f, 8 * ((size_t)n + 1)); g.in_src = rd(f, 4 * (size_t)E);
    g.edge_cls = rd(f, (size_t)E); g.thread_prev = rd(f, 4 * (size_t)n);
    g.thread_id = rd(f, 4 * (size_t)n); g.dur = rd(f, 8 * (size_t)n); g.gap = rd(f, 8 * (size_t)n);
    g.node_cls = rd(f, 2 * (size_t)n);
    ddo_variants vs;
    vs.n_variants = V; vs.n_cls = C; vs.edge_words = K;
    vs.scale = rd(f, 8 * (size_t)C * V); vs.rm_bits = rd(f, 4 * (size_t)n * W);
    vs.edge_on = rd(f, 8 * (size_t)V * K);
    fclose(f);
    FILE *o = fopen(argv[2], "wb");
    int32_t *vl = malloc(4 * (size_t)V);
    for (int32_t v = 0; v < V; v++) vl[v] = v;
    size_t cells = (size_t)V * (n > 0 ? n : 1);
    int64_t *S = malloc(8 * cells), *F = malloc(8 * cells), *M = malloc(8 * (size_t)V),
            *nb = malloc(8 * (size_t)V);
    for (int mode = 0; mode < 2; mode++)
        for (int tie = 0; tie < 3; tie++)
            for (int w = 1; w <= 3; w += 2) {
                int rc = ddo_run(&g, &vs, vl, V, mode, tie, S, F, M, nb, w);
                if (rc) { fprintf(stderr, "oracle status %d\n", rc); return 3; }
                fwrite(S, 8, (size_t)V * n, o);
                fwrite(F, 8, (size_t)V * n, o);
                fwrite(M, 8, (size_t)V, o);
            }
    int32_t *lv = malloc(4 * (size_t)(n > 0 ? n : 1)), *ph = malloc(4 * (size_t)(n > 0 ? n : 1));
    if (ddo_steps(&g, ~0ull, lv, ph)) return 4;
    fwrite(lv, 4, (size_t)n, o);
    fwrite(ph, 4, (size_t)n, o);
    fclose(o);
    free(vl); free(S); free(F); free(M); free(nb); free(lv); free(ph);
    free((void *)g.in_ptr); free((void *)g.in_src); free((void *)g.edge_cls);
    free((void *)g.thread_prev); free((void *)g.thread_id); free((void *)g.dur);
    free((void *)g.gap); free((void *)g.node_cls); free((void *)vs.scale);
    free((void *)vs.rm_bits); free((void *)vs.edge_on);
    printf("ok\n");
    return 0;
}

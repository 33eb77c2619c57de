// Host-side checks of the C-ABI under AddressSanitizer and UBSan, without a
// GPU: argument validation, error reporting, and the clean-up paths taken
// when the first device call fails.  The device passes are replaced by stubs
// (this program links the API layer alone); with no GPU present every call
// that gets past its argument checks fails at its first HIP call, so the
// stubs are never reached.  Exit status 0 = every check held.
#include <stdio.h>
#include <string.h>

#include <thread>

#include "dd_internal.h"

namespace dd {
#define STUB return hipErrorNoDevice
hipError_t scan_exclusive(const int64_t *, int64_t *, int64_t, hipStream_t) { STUB; }
hipError_t launch_validate_nodes(const dd_graph *, const int64_t *, int32_t *, int32_t *,
                                 uint32_t *, LoadStats *, hipStream_t) { STUB; }
hipError_t launch_validate_edges(const dd_graph *, const int64_t *, const int32_t *,
                                 const uint8_t *, const int32_t *, uint32_t *, hipStream_t) { STUB; }
hipError_t launch_rank_tiles(const dd_graph *, int32_t *, int32_t *, int32_t *, int64_t *,
                             uint32_t *, hipStream_t) { STUB; }
hipError_t launch_rank_chains(const dd_graph *, const int32_t *, int32_t *, int32_t *, int32_t *,
                              uint32_t *, hipStream_t) { STUB; }
hipError_t launch_build_order(const dd_graph *, const int32_t *, int64_t *, hipStream_t) { STUB; }
hipError_t launch_cross_edges(dd_graph *, const int64_t *, const int32_t *, const uint8_t *,
                              int64_t *, uint32_t *, LoadStats *, hipStream_t) { STUB; }
hipError_t launch_cross_fill(dd_graph *, const int64_t *, const int32_t *, const uint8_t *,
                             hipStream_t) { STUB; }
dd_status levelize_device(const dd_graph *, uint64_t, int32_t, dd_sched *, hipStream_t, char *msg,
                          size_t len) {
    snprintf(msg, len, "no device");
    return DD_EHIP;
}
hipError_t launch_build_scale_table(const dd_ratio *, int32_t, int32_t, ScaleEntry *, uint32_t *,
                                    hipStream_t) { STUB; }
hipError_t launch_simulate(const dd_graph *, const dd_sched *, const dd_variants *, int64_t *,
                           int64_t *, int64_t *, int, hipStream_t) { STUB; }
hipError_t simulate_noalloc(const dd_graph *, const dd_sched *, const dd_variants *, int64_t *,
                            int64_t *, int64_t *, hipStream_t, size_t *need, size_t *limit) {
    *need = 0;
    *limit = 0;
    STUB;
}
int split_width(const dd_sched *, const dd_variants *) { return 0; }
hipError_t launch_split(const dd_graph *, const dd_sched *, const dd_variants *, int64_t *, int64_t *,
                        int64_t *, int, hipStream_t) { STUB; }
void split_set_polls(int32_t) {}
hipError_t launch_breakdown(const dd_graph *, const dd_variants *, const uint8_t *, const int64_t *,
                            const int64_t *, int64_t *, int32_t *, int64_t *, hipStream_t) { STUB; }
hipError_t build_event_lists(const dd_graph *, EventLists *, hipStream_t) { STUB; }
void free_event_lists(EventLists *ev, hipStream_t) { *ev = EventLists(); }
hipError_t launch_sim_event(const dd_graph *, const EventLists &, const dd_variants *, int32_t,
                            const uint8_t *, const int32_t *, int32_t *, int64_t *, int64_t *,
                            int64_t *, int64_t *, uint32_t *, hipStream_t) { STUB; }
}  // namespace dd

static int g_bad = 0;
#define EXPECT(cond, what)                                                  \
    do {                                                                    \
        if (!(cond)) {                                                      \
            fprintf(stderr, "FAILED: %s (line %d)\n", what, __LINE__);      \
            g_bad++;                                                        \
        }                                                                   \
    } while (0)

static bool has_msg() { return dd_last_error() && dd_last_error()[0] != 0; }

int main() {
    // status names
    const char *names[] = {"DD_OK", "DD_EINVAL", "DD_ECYCLE", "DD_ECHAIN", "DD_ERANGE",
                           "DD_ENOMEM", "DD_EHIP", "DD_EMISMATCH", "DD_ELIMIT"};
    for (int i = 0; i < 9; i++) EXPECT(strcmp(dd_status_str((dd_status)i), names[i]) == 0, "status name");
    EXPECT(strcmp(dd_status_str((dd_status)99), "DD_UNKNOWN") == 0, "unknown status");

    // graph load: argument checks
    int64_t ptr[4] = {0, 0, 1, 1};
    int32_t src[1] = {0}, prev[3] = {-1, 0, -1}, tid[3] = {0, 0, 1};
    int64_t dur[3] = {5, 6, 7}, gap[3] = {1, 0, 0};
    dd_graph *g = (dd_graph *)0x1;
    EXPECT(dd_graph_load(3, 2, ptr, src, nullptr, prev, tid, dur, gap, nullptr, nullptr, nullptr) == DD_EINVAL, "out NULL");
    EXPECT(dd_graph_load(-1, 2, ptr, src, nullptr, prev, tid, dur, gap, nullptr, nullptr, &g) == DD_EINVAL && g == nullptr, "n < 0");
    EXPECT(has_msg(), "message after n < 0");
    EXPECT(dd_graph_load(3, 0, ptr, src, nullptr, prev, tid, dur, gap, nullptr, nullptr, &g) == DD_EINVAL, "n_threads < 1");
    EXPECT(dd_graph_load(3, 2, nullptr, src, nullptr, prev, tid, dur, gap, nullptr, nullptr, &g) == DD_EINVAL, "in_ptr NULL");
    EXPECT(dd_graph_load(3, 2, ptr, src, nullptr, nullptr, tid, dur, gap, nullptr, nullptr, &g) == DD_EINVAL, "thread_prev NULL");
    EXPECT(dd_graph_load(3, 2, ptr, src, nullptr, prev, tid, nullptr, gap, nullptr, nullptr, &g) == DD_EINVAL, "dur NULL");
    // a valid graph: fails at the first device call, and cleans up
    dd_status st = dd_graph_load(3, 2, ptr, src, nullptr, prev, tid, dur, gap, nullptr, nullptr, &g);
    EXPECT(st == DD_EHIP || st == DD_ENOMEM, "no device: load reports a HIP failure");
    EXPECT(g == nullptr && has_msg(), "no handle and a message after a failed load");
    st = dd_graph_load(0, 1, ptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &g);
    EXPECT(st == DD_EHIP || st == DD_ENOMEM, "empty graph without device");
    EXPECT(dd_graph_load_ex(3, 2, ptr, src, nullptr, prev, tid, dur, gap, nullptr, 2u, nullptr, &g) == DD_EINVAL && g == nullptr, "unknown load flag");
    st = dd_graph_load_ex(3, 2, ptr, src, nullptr, prev, tid, dur, gap, nullptr, DD_LOAD_SHARED_THREADS, nullptr, &g);
    EXPECT((st == DD_EHIP || st == DD_ENOMEM) && g == nullptr, "shared-thread load without device");

    // levelize / transforms / simulate argument checks
    dd_sched *sch = (dd_sched *)0x1;
    dd_variants *var = (dd_variants *)0x1;
    EXPECT(dd_levelize(nullptr, ~0ull, DD_PHASES, nullptr, &sch, nullptr) == DD_EINVAL && sch == nullptr, "levelize NULL graph");
    EXPECT(dd_levelize(nullptr, ~0ull, DD_PHASES, nullptr, nullptr, nullptr) == DD_EINVAL, "levelize out NULL");
    EXPECT(dd_apply_transforms(nullptr, 4, 1, nullptr, nullptr, nullptr, nullptr, &var) == DD_EINVAL && var == nullptr, "transforms NULL graph");
    EXPECT(dd_apply_transforms(nullptr, 4, 1, nullptr, nullptr, nullptr, nullptr, nullptr) == DD_EINVAL, "transforms out NULL");
    int64_t dummy[4];
    EXPECT(dd_simulate_batch(nullptr, nullptr, nullptr, dummy, nullptr, dummy, nullptr) == DD_EINVAL, "simulate NULL handles");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, 3, nullptr) == DD_EINVAL, "width 3 rejected");
    EXPECT(strstr(dd_last_error(), "variants_per_wg") != nullptr, "width message");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, 32, nullptr) == DD_EINVAL, "width 32 rejected");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, 16, nullptr) == DD_EINVAL, "width 16 NULL handles");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, -3, nullptr) == DD_EINVAL, "width -3 rejected");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, -16, nullptr) == DD_EINVAL, "width -16 rejected");
    EXPECT(dd_simulate_batch_vs(nullptr, nullptr, nullptr, dummy, nullptr, dummy, -8, nullptr) == DD_EINVAL, "width -8 NULL handles");
    {
        int32_t w = 0;
        EXPECT(dd_simulate_plan(nullptr, nullptr, &w) == DD_EINVAL && has_msg(), "plan of NULL handles");
    }
    dd_set_lookback_polls(0);
    dd_set_lookback_polls(-1);
    EXPECT(dd_runtime_breakdown(nullptr, nullptr, nullptr, dummy, dummy, dummy, nullptr) == DD_EINVAL, "breakdown NULL handles");
    EXPECT(dd_simulate_batch_noalloc(nullptr, nullptr, nullptr, dummy, nullptr, dummy, nullptr) == DD_EINVAL, "no-alloc NULL handles");
    EXPECT(dd_simulate_policy(nullptr, nullptr, 0, nullptr, nullptr, dummy, nullptr, dummy, nullptr) == DD_EINVAL, "policy NULL handles");
    EXPECT(strstr(dd_last_error(), "NULL handle") != nullptr, "NULL handle message");
    EXPECT(dd_sched_task_steps(nullptr, nullptr, nullptr) == DD_EINVAL, "steps NULL");
    int64_t a, b, c, d;
    EXPECT(dd_sched_info(nullptr, &a, &b, &c, &d) == DD_EINVAL, "info NULL");
    dd_graph_free(nullptr);
    dd_sched_free(nullptr);
    dd_variants_free(nullptr);
    st = dd_release_cache();
    EXPECT(st == DD_OK || st == DD_EHIP, "release cache");

    // error messages are per host thread
    std::thread t1([] { (void)dd_graph_load(-5, 1, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr); });
    t1.join();
    EXPECT(dd_levelize(nullptr, 0, 7, nullptr, &sch, nullptr) == DD_EINVAL, "bad mode");
    char mine[512];
    snprintf(mine, sizeof(mine), "%s", dd_last_error());
    std::thread t2([] { (void)dd_simulate_batch_vs(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 5, nullptr); });
    t2.join();
    EXPECT(strcmp(mine, dd_last_error()) == 0, "thread-local message");
    if (g_bad == 0) printf("ALL OK\n");
    return g_bad ? 1 : 0;
}

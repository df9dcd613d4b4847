// Host-side thread-safety check of liblinattn: many threads call the host
// entry points at once (boundary selection, checkpoint rows, workspace
// sizes, kernel-form queries, argument validation with its per-thread
// error message, the static-workspace size check, the trace hook).  Built with ThreadSanitizer over a
// host-only build of the library; no GPU is needed, since every prefill
// call here is refused on the host before any launch.  Exit status 0 and
// no ThreadSanitizer report mean no data race was seen.
#include <cstdio>
#include <cstring>
#include <thread>
#include <vector>

#include "linattn.h"

static int worker(int t) {
    int bad = 0;
    for (int it = 0; it < 2000; ++it) {
        const int64_t n = 1 + (it * 37 + t * 101) % 9000, C = 16 << (it % 5);
        int64_t b = -1;
        if (strict_prefix_boundary(n, C, n, &b) != LA_OK || b != C * ((n - 1) / C)) ++bad;
        int32_t cu[4] = {0, (int32_t)n, (int32_t)(n + 300), (int32_t)(n + 300 + t)};
        int64_t start[3] = {0, C, 2 * C};
        int32_t offs[3];
        int64_t rows = -1;
        if (la_checkpoint_rows(3, cu, start, (int32_t)C, offs, &rows) != LA_OK || rows < 0) ++bad;
        la_shape s{};
        s.n_seqs = 3;
        s.n_heads = 1 + t % 8;
        s.dk = (it & 1) ? 128 : 64;
        s.dv = (it & 2) ? 128 : 64;
        s.chunk = 64;
        s.ckpt_interval = (int32_t)C;
        s.io_dtype = (it & 4) ? LA_BF16 : LA_F32;
        s.variant = LA_GDR_LITERAL;
        s.scale = 1.0f;
        if (la_prefill_workspace_bytes(&s, cu[3]) == 0) ++bad;
        if (la_prefill_form(&s) == LA_FORM_NONE) ++bad;
        // a refused call: the message read back is this thread's own
        s.n_seqs = -(t + 1);
        const la_status st = la_prefill(&s, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, cu, nullptr,
                                        nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr);
        char want[32];
        snprintf(want, sizeof want, "n_seqs=%d", -(t + 1));
        if (st != LA_ERR_INVALID_ARG || !strstr(la_last_error_message(), want)) ++bad;
        // the static-workspace entry point refuses a call larger than its array
        s.n_seqs = 1;
        s.io_dtype = LA_BF16;
        int32_t big[2] = {0, 2000000 + t};
        if (la_prefill_paged_noalloc(&s, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, big, nullptr,
                                     nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) != LA_ERR_WORKSPACE)
            ++bad;
        void *ev[4] = {nullptr, nullptr, nullptr, nullptr};
        la_trace_set_events((it & 1) ? ev : nullptr, (it & 1) ? 4 : 0);
    }
    la_trace_set_events(nullptr, 0);
    return bad;
}

int main() {
    const int n = 8;
    std::vector<std::thread> th;
    std::vector<int> bad(n, 0);
    for (int t = 0; t < n; ++t) th.emplace_back([t, &bad]() { bad[t] = worker(t); });
    for (auto &x : th) x.join();
    int total = 0;
    for (int b : bad) total += b;
    printf("host threads: %d threads, %d mismatches\n", n, total);
    return total == 0 ? 0 : 1;
}

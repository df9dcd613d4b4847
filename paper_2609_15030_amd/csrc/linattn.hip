// C ABI of the strict-prefix linear-attention prefill library (gfx950).
// Host side: argument validation, the chunk plan's sizes, workspace carving
// and launches.  Kernels live in the headers included below.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "linattn.h"
#include "la_common.h"
#include "gdr_prep.h"
#include "gdr_scan.h"
#include "gdr_group.h"
#include "gdr_scan_pair.h"
#include "gdr_out.h"
#include "gdr_decode.h"
#include "paged.h"
#include "hybrid.h"

namespace {

thread_local char g_msg[512] = "";
thread_local void *g_trace[4] = {nullptr, nullptr, nullptr, nullptr};
thread_local int g_trace_n = 0;

la_status fail(la_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
    va_end(ap);
    return s;
}

la_status hip_check(const char *what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(LA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return LA_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

constexpr size_t kRegionAlign = 256;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Scan kernel form: 1 = one wave per 16-column tile, 4 = DK/32 waves sharing
// the tile's state rows.  The single-wave form has the shorter chain; with
// fp32 operands at dk = 128 it does not fit the register file, so that case
// splits dk.  LA_SCAN_WAVES=1|4 overrides the choice (for tuning).
int scan_variant(bool f32, int dk) {
    static const int forced = [] {
        const char *e = getenv("LA_SCAN_WAVES");
        return e ? atoi(e) : 0;
    }();
    if (forced == 1 || forced == 4) return forced;
    return (f32 && dk == 128) ? 4 : 1;
}

size_t io_size(int32_t dtype) { return dtype == LA_BF16 ? 2 : 4; }

// Whether a call that runs the scan and output stages together uses the
// single-wave scan's output wave (one kernel) instead of the split output
// kernel or the workgroup scan; all give identical bits.  The
// scan-with-output workgroup holds two waves with a large register file
// each, so few of them fit on a CU, and each is one sequential chain: a
// launch that needs more rounds of residency than it has chains per round
// runs its later chains after the first ones end.  fp32 operands use it
// only while every workgroup is resident at once; bf16 up to two rounds
// (on a 16-sequence, 8-head batch of 1,024 tiles with 512 resident it beat
// both the split kernels, whose state and U make a round trip through HBM,
// and the workgroup scan, bound by its CU's LDS bandwidth).
// LA_SCAN_OUTPUT=0 selects the split kernels (for measurement).
bool output_waves_on() {
    static const bool on = [] {
        const char *e = getenv("LA_SCAN_OUTPUT");
        return !(e && atoi(e) == 0);
    }();
    return on;
}

template <typename T, int DK, int DV>
bool scan_with_output(int64_t blocks) {
    if (!output_waves_on()) return false;
    static int64_t capacity[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return false;
    }
    if (capacity[dev] == 0) {
        int per_cu = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, la::gdr_scan1o_kernel<T, DK, DV>, 128, 0) !=
                hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        capacity[dev] = (int64_t)per_cu * cus;
    }
    const int64_t rounds = sizeof(T) == 2 ? 2 : 1;
    return blocks <= rounds * capacity[dev];
}

// Workgroups of `kernel` (launched with `threads` lanes) resident on the
// current device at once; cached per device and caller slot.  0 when the
// runtime cannot say.
template <typename K>
int64_t resident_capacity(K kernel, int threads, int slot) {
    static int64_t cache[4][64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64 || slot < 0 || slot >= 4) {
        (void)hipGetLastError();
        return 0;
    }
    if (cache[slot][dev] == 0) {
        int per_cu = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
            (void)hipGetLastError();
            return 0;
        }
        cache[slot][dev] = (int64_t)per_cu * cus;
    }
    return cache[slot][dev];
}

// Whether a bf16 call with the scan and output stages runs the scan with
// output wave over pairs of column tiles (gdr_scan2o_kernel) instead of one
// tile per workgroup: when the one-tile workgroups do not all fit at once
// but the pair workgroups fit in two rounds.  Several scan workgroups then
// share each CU, whose load path bounds their chunk steps, and a pair moves
// half the operand bytes per tile (16-sequence, 8-head varlen batch:
// 1,024 one-tile or 512 pair workgroups).  LA_SCAN_PAIR=1|0 forces the
// choice (for measurement).
template <typename T, int DK, int DV>
bool scan_by_pairs(int64_t blocks1, int64_t blocks2) {
    static const int forced = [] {
        const char *e = getenv("LA_SCAN_PAIR");
        return e ? atoi(e) : -1;
    }();
    if (forced == 0 || forced == 1) return forced == 1;
    if (!output_waves_on()) return false;
    const int64_t cap1 = resident_capacity(la::gdr_scan1o_kernel<T, DK, DV>, 128, 0);
    const int64_t cap2 = resident_capacity(la::gdr_scan2o_kernel<T, DK, DV>, 128, 1);
    return cap1 > 0 && cap2 > 0 && blocks1 > cap1 && blocks2 <= 2 * cap2;
}

// Whether a single-level bf16 scan runs as one workgroup per (sequence,
// head) chain (the chunk operands shared through LDS, output waves beside
// the scan waves) instead of one wave per 16-column tile.  By default the
// workgroup form serves the calls that include the output stage and have
// more tiles than the per-tile scan with output wave takes (see
// scan_with_output); the split kernels' output would make a round trip
// through HBM.  LA_SCAN_GROUP=1|0 forces the choice (for measurement).
bool scan_by_group(bool tile_scan_with_output, bool output_stage) {
    static const int forced = [] {
        const char *e = getenv("LA_SCAN_GROUP");
        return e ? atoi(e) : -1;
    }();
    if (forced == 0 || forced == 1) return forced == 1;
    return output_stage && !tile_scan_with_output && output_waves_on();
}

// Chunks per segment of the two-level scan (1 = single-level).  A segment
// must divide a checkpoint interval's chunks, so every checkpoint position is
// a segment boundary and a resume from a checkpoint sees the same segments
// (and computes bit-identical states) as the run that wrote it; for the same
// reason the choice depends on the interval only, never on the lengths.  The
// largest such divisor up to 16 balances the two parallel levels against the
// sequential combine.  Intervals of fewer than 8 chunks keep the
// single-level scan: there a segment's map costs more than the chunks it
// replaces.  bf16 operands only.  LA_SCAN_LEVELS=1|2 forces one form (for
// tuning).
int seg_chunks(const la_shape *s) {
    static const int forced = [] {
        const char *e = getenv("LA_SCAN_LEVELS");
        return e ? atoi(e) : 0;
    }();
    if (forced == 1 || s->io_dtype != LA_BF16) return 1;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    if (forced != 2 && cps < 8) return 1;
    for (int m = std::min(cps, 16); m >= 2; --m)
        if (cps % m == 0) return m;
    return 1;
}

bool shape_supported(const la_shape *s) {
    return (s->dk == 64 || s->dk == 128) && (s->dv == 64 || s->dv == 128) && s->chunk == la::kChunk;
}

la_status check_shape(const la_shape *s) {
    if (!s) return fail(LA_ERR_INVALID_ARG, "shape is NULL");
    if (s->n_seqs < 1 || s->n_seqs > 65535) return fail(LA_ERR_INVALID_ARG, "n_seqs=%d outside [1, 65535]", s->n_seqs);
    if (s->n_heads < 1 || s->n_heads > 65535) return fail(LA_ERR_INVALID_ARG, "n_heads=%d outside [1, 65535]", s->n_heads);
    if (s->ckpt_interval < 1) return fail(LA_ERR_INVALID_ARG, "ckpt_interval=%d < 1", s->ckpt_interval);
    if (s->io_dtype != LA_F32 && s->io_dtype != LA_BF16) return fail(LA_ERR_INVALID_ARG, "io_dtype=%d", s->io_dtype);
    if (s->variant != LA_GDR_LITERAL && s->variant != LA_GDR_DECAYED_DELTA)
        return fail(LA_ERR_INVALID_ARG, "variant=%d", s->variant);
    if (!std::isfinite(s->scale)) return fail(LA_ERR_INVALID_ARG, "scale is not finite");
    if (s->dk < 1 || s->dv < 1 || s->chunk < 1) return fail(LA_ERR_INVALID_ARG, "dk, dv, chunk must be >= 1");
    if (!shape_supported(s))
        return fail(LA_ERR_UNSUPPORTED, "dk=%d dv=%d chunk=%d not built (dk, dv in {64, 128}, chunk 64)",
                    s->dk, s->dv, s->chunk);
    return LA_OK;
}

struct WsPlan {
    size_t w, kt, ut, g, sc, u, pm, qf;      // byte offsets of each region
    size_t phi, segr, segd, segst;           // two-level scan regions (seg_m >= 2)
    int seg_m;
    size_t total;
};

WsPlan plan_workspace(const la_shape *s, int64_t total_tokens) {
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    const int64_t slots = la::total_slots(total_tokens, s->n_seqs, s->ckpt_interval, cps);
    const size_t sh = (size_t)slots * s->n_heads;
    const size_t io = io_size(s->io_dtype);
    WsPlan p;
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t at = off; off = round_up(off + bytes, kRegionAlign); return at; };
    p.w = take(sh * la::kChunk * s->dk * io);
    p.kt = take(sh * s->dk * la::kChunk * io);
    p.ut = take(sh * la::kChunk * s->dv * io);
    p.g = take(sh * la::kChunk * sizeof(float));
    p.sc = take(sh * (size_t)s->dk * s->dv * io);
    p.u = take(sh * la::kChunk * s->dv * io);
    p.pm = take(sh * la::kChunk * la::kChunk * io);
    p.qf = take(sh * la::kChunk * s->dk * io);
    p.seg_m = seg_chunks(s);
    p.phi = p.segr = p.segd = p.segst = 0;
    if (p.seg_m > 1) {
        const int64_t seg_slots = la::total_slots(total_tokens, s->n_seqs, s->ckpt_interval * (int64_t)p.seg_m, cps);
        const size_t ssh = (size_t)seg_slots * s->n_heads;
        p.phi = take(ssh * s->dk * s->dk * io);
        p.segr = take(ssh * s->dk * s->dv * sizeof(float));
        p.segd = take(ssh * sizeof(float));
        p.segst = take(ssh * s->dk * s->dv * sizeof(float));
    }
    p.total = std::max<size_t>(off, kRegionAlign);
    return p;
}

struct PrefillCall {
    const la_shape *shape;
    const void *q, *k, *v;
    const float *g, *beta;
    const int32_t *cu_dev, *cu_host;
    const int64_t *start_dev, *start_host;   // null for a cold prefill
    const float *state_in;                   // null for a cold prefill
    void *o;
    float *final_state, *ckpt_out;
    const int32_t *ckpt_off_dev, *ckpt_off_host;
    void *workspace;
    size_t ws_bytes;
    hipStream_t stream;
    uint32_t stages = LA_STAGE_ALL;
    const la_pages *pages = nullptr;         // paged checkpoints / starting states
};

template <typename T, int DK, int DV>
la_status launch_out(const PrefillCall &c, const la::Workspace &ws, int64_t max_chunks, bool trace) {
    const la_shape *s = c.shape;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    if (trace) (void)hipEventRecord((hipEvent_t)g_trace[2], c.stream);
    if (max_chunks > 0 && (c.stages & LA_STAGE_OUTPUT)) {
        la::OutArgs oa{c.o, c.cu_dev, s->n_seqs, s->n_heads, s->ckpt_interval, cps,
                       (int32_t)max_chunks, s->scale, ws,
                       la::chunk_major_map(s->n_seqs, s->n_heads, max_chunks) ? 1 : 0};
        const int64_t blocks = la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks);
        hipLaunchKernelGGL((la::gdr_out_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(4 * DV), 0, c.stream, oa);
        if (la_status e = hip_check("output launch")) return e;
    }
    if (trace) (void)hipEventRecord((hipEvent_t)g_trace[3], c.stream);
    return LA_OK;
}

// Two-level scan: segment maps (all segments at once), the sequential
// combine over segments, then every segment replayed from its entering
// state; then the output kernel.
template <typename T, int DK, int DV>
la_status launch_two_level(const PrefillCall &c, const WsPlan &p, la::ScanArgs sa, int64_t max_chunks,
                           bool trace) {
    const la_shape *s = c.shape;
    char *base = (char *)c.workspace;
    sa.seg_m = p.seg_m;
    sa.max_seg = (int32_t)((max_chunks + p.seg_m - 1) / p.seg_m);
    sa.seg.phi = base + p.phi;
    sa.seg.r = (float *)(base + p.segr);
    sa.seg.d = (float *)(base + p.segd);
    sa.seg.state = (float *)(base + p.segst);
    constexpr int NT = DV / 16;
    const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
    const int64_t units = pairs * sa.max_seg;
    if (units > 0) {
        hipLaunchKernelGGL((la::gdr_group_kernel<T, DK, DV, la::kGroupTrans>), dim3((unsigned)units),
                           dim3(64 * la::group_scan_waves<DK, DV, la::kGroupTrans>()), 0, c.stream, sa);
        if (la_status e = hip_check("segment map launch")) return e;
    }
    hipLaunchKernelGGL((la::gdr_seg_combine_kernel<T, DK, DV>), dim3((unsigned)(8 * NT * ((pairs + 7) / 8))),
                       dim3(64), 0, c.stream, sa);
    if (la_status e = hip_check("segment combine launch")) return e;
    // the replay's output waves produce the output when the call includes
    // the output stage; otherwise the split output kernel reads the states
    // and U the replay leaves in the workspace
    const bool out_stage = (c.stages & LA_STAGE_OUTPUT) != 0 && output_waves_on();
    if (units > 0) {
        if (out_stage)
            hipLaunchKernelGGL((la::gdr_group_kernel<T, DK, DV, la::kGroupReplay, true>), dim3((unsigned)units),
                               dim3(128 * la::kGroupWaves), 0, c.stream, sa);
        else
            hipLaunchKernelGGL((la::gdr_group_kernel<T, DK, DV, la::kGroupReplay>), dim3((unsigned)units),
                               dim3(64 * la::kGroupWaves), 0, c.stream, sa);
        if (la_status e = hip_check("segment replay launch")) return e;
    }
    return launch_out<T, DK, DV>(c, sa.ws, out_stage ? 0 : max_chunks, trace);
}

// Ranks the (sequence, head) chains for dispatch, longest first (equal
// lengths keep sequence order), so the workgroups each CU receives mix long
// and short chains.  Batches of more than kChainOrderMax chains, or of one
// sequence, keep the natural order.
void order_chains(const PrefillCall &c, la::ChainOrder &order) {
    const la_shape *s = c.shape;
    const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
    order.n = 0;
    if (s->n_seqs < 2 || pairs > la::kChainOrderMax) return;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    int64_t nch[la::kChainOrderMax];
    for (int i = 0; i < s->n_seqs; ++i)
        nch[i] = la::n_chunks((int64_t)c.cu_host[i + 1] - c.cu_host[i], s->ckpt_interval, cps);
    int32_t idx[la::kChainOrderMax];
    for (int64_t k = 0; k < pairs; ++k) idx[k] = (int32_t)k;
    const int H = s->n_heads;
    std::stable_sort(idx, idx + pairs, [&](int32_t x, int32_t y) { return nch[x / H] > nch[y / H]; });
    for (int64_t k = 0; k < pairs; ++k) order.pair[k] = (uint16_t)idx[k];
    order.n = (int32_t)pairs;
}

template <typename T, int DK, int DV>
la_status launch_prefill(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    const la_shape *s = c.shape;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    char *base = (char *)c.workspace;
    la::Workspace ws;
    ws.w = base + p.w;
    ws.kt = base + p.kt;
    ws.ut = base + p.ut;
    ws.g = (float *)(base + p.g);
    ws.sc = base + p.sc;
    ws.u = base + p.u;
    ws.p = base + p.pm;
    ws.qf = base + p.qf;

    const bool trace = g_trace_n >= 4;
    if (trace) (void)hipEventRecord((hipEvent_t)g_trace[0], c.stream);
    (void)hipGetLastError();

    if (max_chunks > 0 && (c.stages & LA_STAGE_PREPARE)) {
        la::PrepArgs pa{c.q, c.k, c.v, c.g, c.beta, c.cu_dev, s->n_seqs, s->n_heads, s->ckpt_interval, cps,
                        s->variant, (int32_t)max_chunks, ws,
                        la::chunk_major_map(s->n_seqs, s->n_heads, max_chunks) ? 1 : 0};
        const int64_t blocks = la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks);
        hipLaunchKernelGGL((la::gdr_prep_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(256), 0, c.stream, pa);
        if (la_status e = hip_check("chunk preparation launch")) return e;
    }
    if (trace) (void)hipEventRecord((hipEvent_t)g_trace[1], c.stream);
    if (c.stages & LA_STAGE_SCAN) {
        la::ScanArgs sa{c.cu_dev, c.state_in, c.final_state, c.ckpt_out, c.ckpt_off_dev,
                        s->n_seqs, s->n_heads, s->ckpt_interval, cps, ws, 1, 0, {},
                        c.o, s->scale, {}};
        if (c.pages) {
            sa.pg.pool = c.pages->pool;
            sa.pg.ckpt_ids = c.pages->ckpt_page_ids;
            sa.pg.state_ids = c.pages->state_page_ids;
            sa.pg.err = c.pages->err_count;
            sa.pg.n_pages = (int32_t)c.pages->n_pages;
        }
        constexpr int NT = DV / 16;
        const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
        const int64_t blocks = 8 * NT * ((pairs + 7) / 8);
        order_chains(c, sa.order);
        if constexpr (sizeof(T) == 2) {
            if (p.seg_m > 1) return launch_two_level<T, DK, DV>(c, p, sa, max_chunks, trace);
        }
        const bool out_stage = (c.stages & LA_STAGE_OUTPUT) != 0;
        if constexpr (sizeof(T) == 2) {
            const int64_t blocks2 = 8 * (NT / la::kPairTiles) * ((pairs + 7) / 8);
            if (out_stage && scan_variant(false, DK) == 1 && scan_by_pairs<T, DK, DV>(blocks, blocks2)) {
                hipLaunchKernelGGL((la::gdr_scan2o_kernel<T, DK, DV>), dim3((unsigned)blocks2), dim3(128), 0,
                                   c.stream, sa);
                if (la_status e = hip_check("inter-chunk scan launch")) return e;
                return launch_out<T, DK, DV>(c, ws, 0, trace);
            }
        }
        const bool with_out = scan_variant(sizeof(T) == 4, DK) == 1 && out_stage && scan_with_output<T, DK, DV>(blocks);
        if constexpr (sizeof(T) == 2) {
            // the workgroup scan stands in for the single-wave form only (the
            // dk-split scan sums its partial products in another order)
            if (scan_variant(false, DK) == 1 && scan_by_group(with_out, out_stage)) {
                // one workgroup per (sequence, head) chain: 4 scan waves, and
                // 4 output waves when the call includes the output stage
                sa.seg_m = 1;
                sa.max_seg = 1;
                if (out_stage)
                    hipLaunchKernelGGL((la::gdr_group_kernel<T, DK, DV, la::kGroupScan, true>), dim3((unsigned)pairs),
                                       dim3(128 * la::kGroupWaves), 0, c.stream, sa);
                else
                    hipLaunchKernelGGL((la::gdr_group_kernel<T, DK, DV, la::kGroupScan>), dim3((unsigned)pairs),
                                       dim3(64 * la::kGroupWaves), 0, c.stream, sa);
                if (la_status e = hip_check("inter-chunk scan launch")) return e;
                return launch_out<T, DK, DV>(c, ws, 0, trace);
            }
        }
        if (with_out) {
            // the scan's output wave produces the output: no output launch
            hipLaunchKernelGGL((la::gdr_scan1o_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(128), 0,
                               c.stream, sa);
            if (la_status e = hip_check("inter-chunk scan launch")) return e;
            return launch_out<T, DK, DV>(c, ws, 0, trace);
        }
        if (scan_variant(sizeof(T) == 4, DK) == 1)
            hipLaunchKernelGGL((la::gdr_scan1_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(64), 0,
                               c.stream, sa);
        else
            hipLaunchKernelGGL((la::gdr_scan_kernel<T, DK, DV>), dim3((unsigned)blocks),
                               dim3(64 * la::ScanGeom<DK>::NW), 0, c.stream, sa);
        if (la_status e = hip_check("inter-chunk scan launch")) return e;
    }
    return launch_out<T, DK, DV>(c, ws, max_chunks, trace);
}

template <typename T>
la_status dispatch_dims(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    const int dk = c.shape->dk, dv = c.shape->dv;
    if (dk == 64 && dv == 64) return launch_prefill<T, 64, 64>(c, p, max_chunks);
    if (dk == 64 && dv == 128) return launch_prefill<T, 64, 128>(c, p, max_chunks);
    if (dk == 128 && dv == 64) return launch_prefill<T, 128, 64>(c, p, max_chunks);
    if (dk == 128 && dv == 128) return launch_prefill<T, 128, 128>(c, p, max_chunks);
    return fail(LA_ERR_UNSUPPORTED, "dk=%d dv=%d", dk, dv);
}

la_status run_prefill(const PrefillCall &c) {
    if (la_status e = check_shape(c.shape)) return e;
    const la_shape *s = c.shape;
    const bool resume = c.start_host != nullptr || c.start_dev != nullptr;
    if (c.stages == 0 || (c.stages & ~LA_STAGE_ALL)) return fail(LA_ERR_INVALID_ARG, "stages=%u", c.stages);
    if (!resume && c.state_in) return fail(LA_ERR_INVALID_ARG, "state_in given without start positions");
    const int64_t C = s->ckpt_interval;
    const int cps = la::chunks_per_interval(s->ckpt_interval);

    if (!c.cu_dev || !c.cu_host) return fail(LA_ERR_INVALID_ARG, "cu_seqlens_dev and cu_seqlens_host are required");
    if (c.cu_host[0] != 0) return fail(LA_ERR_INVALID_ARG, "cu_seqlens[0]=%d, must be 0", c.cu_host[0]);
    int64_t max_chunks = 0;
    for (int i = 0; i < s->n_seqs; ++i) {
        const int64_t len = (int64_t)c.cu_host[i + 1] - c.cu_host[i];
        if (len < 0) return fail(LA_ERR_INVALID_ARG, "cu_seqlens decreases at sequence %d", i);
        if (c.cu_host[i + 1] < 0) return fail(LA_ERR_INVALID_ARG, "cu_seqlens overflows int32");
        max_chunks = std::max(max_chunks, la::n_chunks(len, C, cps));
    }
    const int64_t total = c.cu_host[s->n_seqs];
    if (c.pages) {
        const la_pages *pg = c.pages;
        if (c.state_in || c.ckpt_out) return fail(LA_ERR_INVALID_ARG, "internal: paged call with dense state I/O");
        if (pg->n_pages < 0 || pg->n_pages > 0x7fffffff)
            return fail(LA_ERR_INVALID_ARG, "n_pages=%lld", (long long)pg->n_pages);
        if ((pg->ckpt_page_ids || pg->state_page_ids) && (!pg->pool || !aligned16(pg->pool)))
            return fail(LA_ERR_INVALID_ARG, "pages->pool is required (16-byte aligned) with page ids");
        if (pg->state_page_ids && !resume)
            return fail(LA_ERR_INVALID_ARG, "state_page_ids given without start positions");
        if (resume && !pg->state_page_ids)
            return fail(LA_ERR_INVALID_ARG, "state_page_ids are required for a resume");
        if (pg->ckpt_page_ids && (!c.ckpt_off_dev || !c.ckpt_off_host))
            return fail(LA_ERR_INVALID_ARG, "ckpt_offsets_dev and ckpt_offsets_host are required with ckpt_page_ids");
    }
    if (resume) {
        if (!c.start_host || !c.start_dev) return fail(LA_ERR_INVALID_ARG, "start_pos_dev and start_pos_host are required");
        if (!c.state_in && !c.pages) return fail(LA_ERR_INVALID_ARG, "state_in is required for a resume");
        for (int i = 0; i < s->n_seqs; ++i) {
            const int64_t B = c.start_host[i];
            const int64_t len = (int64_t)c.cu_host[i + 1] - c.cu_host[i];
            if (B < 0) return fail(LA_ERR_INVALID_ARG, "start_pos[%d]=%lld < 0", i, (long long)B);
            if (B % C != 0)
                return fail(LA_ERR_MISALIGNED_STATE, "start_pos[%d]=%lld is not a multiple of C=%lld: no checkpoint "
                            "represents that prefix", i, (long long)B, (long long)C);
            if (len == 0)
                return fail(LA_ERR_EMPTY_SUFFIX, "sequence %d has an empty suffix (B = N = %lld): the restored state "
                            "already covers the prompt", i, (long long)B);
            if (B > ((int64_t)1 << 40)) return fail(LA_ERR_INVALID_ARG, "start_pos[%d] too large", i);
        }
    }
    if (max_chunks > 0x7fffffff ||
        la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks) > 0x7fffffff)
        return fail(LA_ERR_INVALID_ARG, "sequence too long for one launch");
    {
        const int m = seg_chunks(s);
        const int64_t units = (int64_t)s->n_seqs * s->n_heads * ((max_chunks + m - 1) / m);
        if (m > 1 && units > 0x7fffffff)
            return fail(LA_ERR_INVALID_ARG, "too many segments for one launch");
    }
    if (total > 0) {
        if (!c.q || !c.k || !c.v || !c.g || !c.beta || !c.o)
            return fail(LA_ERR_INVALID_ARG, "q, k, v, g, beta and o are required");
        if (!aligned16(c.q) || !aligned16(c.k) || !aligned16(c.v) || !aligned16(c.o))
            return fail(LA_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
    }
    if (c.state_in && !aligned16(c.state_in)) return fail(LA_ERR_INVALID_ARG, "state_in must be 16-byte aligned");
    if (c.final_state && !aligned16(c.final_state)) return fail(LA_ERR_INVALID_ARG, "final_state must be 16-byte aligned");
    if (c.ckpt_out) {
        if (!aligned16(c.ckpt_out)) return fail(LA_ERR_INVALID_ARG, "ckpt_out must be 16-byte aligned");
        if (!c.ckpt_off_dev || !c.ckpt_off_host)
            return fail(LA_ERR_INVALID_ARG, "ckpt_offsets_dev and ckpt_offsets_host are required with ckpt_out");
    }
    if (c.ckpt_out || (c.pages && c.pages->ckpt_page_ids)) {
        for (int i = 0; i < s->n_seqs; ++i)
            if (c.ckpt_off_host[i] < 0) return fail(LA_ERR_INVALID_ARG, "ckpt_offsets[%d] < 0", i);
    }
    const WsPlan p = plan_workspace(s, total);
    if (!c.workspace || c.ws_bytes < p.total)
        return fail(LA_ERR_WORKSPACE, "workspace of %zu bytes, %zu required", c.workspace ? c.ws_bytes : 0, p.total);
    if (!aligned16(c.workspace)) return fail(LA_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    // The chunk plan's slot bound, checked on the host before any launch.
    const int64_t slots = la::total_slots(total, s->n_seqs, C, cps);
    for (int i = 0; i < s->n_seqs; ++i) {
        const int64_t len = (int64_t)c.cu_host[i + 1] - c.cu_host[i];
        if (la::slot_base(c.cu_host[i], i, C, cps) + la::n_chunks(len, C, cps) > slots)
            return fail(LA_ERR_INVALID_ARG, "internal: chunk plan exceeds its workspace at sequence %d", i);
    }
    if (p.seg_m > 1) {
        const int64_t K = C * p.seg_m;
        const int64_t seg_slots = la::total_slots(total, s->n_seqs, K, cps);
        for (int i = 0; i < s->n_seqs; ++i) {
            const int64_t len = (int64_t)c.cu_host[i + 1] - c.cu_host[i];
            const int64_t nseg = (la::n_chunks(len, C, cps) + p.seg_m - 1) / p.seg_m;
            if (la::slot_base(c.cu_host[i], i, K, cps) + nseg > seg_slots)
                return fail(LA_ERR_INVALID_ARG, "internal: segment plan exceeds its workspace at sequence %d", i);
        }
    }

    if (s->io_dtype == LA_BF16) return dispatch_dims<__bf16>(c, p, max_chunks);
    return dispatch_dims<float>(c, p, max_chunks);
}

template <typename T, int DK, int DV>
la_status launch_decode(const la_shape *s, const la::DecodeArgs &a, hipStream_t stream) {
    const int64_t blocks = (int64_t)s->n_seqs * s->n_heads * (DV / la::kDecodeCols);
    hipLaunchKernelGGL((la::gdr_decode_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(la::kDecodeThreads), 0,
                       stream, a);
    return hip_check("decode launch");
}

template <typename T>
la_status decode_dims(const la_shape *s, const la::DecodeArgs &a, hipStream_t stream) {
    if (s->dk == 64 && s->dv == 64) return launch_decode<T, 64, 64>(s, a, stream);
    if (s->dk == 64 && s->dv == 128) return launch_decode<T, 64, 128>(s, a, stream);
    if (s->dk == 128 && s->dv == 64) return launch_decode<T, 128, 64>(s, a, stream);
    return launch_decode<T, 128, 128>(s, a, stream);
}

// A host-tier pool is pinned host memory mapped into the device's address
// space (hipHostMalloc, or a torch tensor allocated with pin_memory=True):
// the copy kernels read or write it directly over the host link.  Both ends
// of the pool are checked before any launch, so pageable or unmapped memory
// is rejected instead of being dereferenced by a kernel.  Returns the device
// address of the pool's first byte.
la_status host_pool_device_ptr(const float *pool, size_t bytes, float **dev) {
    *dev = nullptr;
    if (!pool) return fail(LA_ERR_INVALID_ARG, "host pool is NULL");
    hipPointerAttribute_t a0{}, a1{};
    const char *last = (const char *)pool + (bytes ? bytes - 1 : 0);
    if (hipPointerGetAttributes(&a0, pool) != hipSuccess || hipPointerGetAttributes(&a1, last) != hipSuccess) {
        (void)hipGetLastError();
        return fail(LA_ERR_INVALID_ARG, "host pool is not pinned, device-mapped host memory");
    }
    if (a0.type != hipMemoryTypeHost || a1.type != hipMemoryTypeHost || !a0.devicePointer || !a1.devicePointer)
        return fail(LA_ERR_INVALID_ARG, "host pool is not pinned, device-mapped host memory");
    if ((const char *)a1.devicePointer - (const char *)a0.devicePointer != last - (const char *)pool)
        return fail(LA_ERR_INVALID_ARG, "host pool does not map to one contiguous device range");
    *dev = (float *)a0.devicePointer;
    return LA_OK;
}

// A pool the kernels read directly: device memory as is, or pinned host
// memory through its device mapping (checked at both ends).  Pageable or
// unknown memory is refused.
la_status resolve_pool(const void *p, size_t bytes, const void **dev, const char *what) {
    *dev = nullptr;
    hipPointerAttribute_t at{};
    if (!p || hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(LA_ERR_INVALID_ARG, "%s is neither device memory nor pinned, device-mapped host memory", what);
    }
    if (at.type == hipMemoryTypeDevice) {
        *dev = p;
        return LA_OK;
    }
    if (at.type == hipMemoryTypeHost) {
        float *d = nullptr;
        if (la_status e = host_pool_device_ptr((const float *)p, bytes, &d)) return e;
        *dev = d;
        return LA_OK;
    }
    return fail(LA_ERR_INVALID_ARG, "%s is neither device memory nor pinned, device-mapped host memory", what);
}

la_status record_done(void *done_event, void *stream) {
    if (done_event && hipEventRecord((hipEvent_t)done_event, (hipStream_t)stream) != hipSuccess)
        return hip_check("completion event record");
    return LA_OK;
}

la_status check_paged(const float *a, const float *b, int64_t n_items, int64_t page_elems, int64_t n_pages,
                      const int32_t *ids) {
    if (n_items < 0 || n_items > 0x7fffffff) return fail(LA_ERR_INVALID_ARG, "n_items=%lld", (long long)n_items);
    if (page_elems <= 0 || page_elems % 4 != 0)
        return fail(LA_ERR_INVALID_ARG, "page_elems=%lld must be a positive multiple of 4", (long long)page_elems);
    if (n_pages < 0 || n_pages > 0x7fffffff) return fail(LA_ERR_INVALID_ARG, "n_pages=%lld", (long long)n_pages);
    if (n_items > 0 && (!a || !b || !ids)) return fail(LA_ERR_INVALID_ARG, "states, pool and page_ids are required");
    if (!aligned16(a) || !aligned16(b)) return fail(LA_ERR_INVALID_ARG, "states and pool must be 16-byte aligned");
    return LA_OK;
}

}  // namespace

extern "C" {

la_status strict_prefix_boundary(int64_t n_tokens, int64_t interval, int64_t available_tokens,
                                 int64_t *boundary_out) {
    if (!boundary_out) return fail(LA_ERR_INVALID_ARG, "boundary_out is NULL");
    if (n_tokens < 1) return fail(LA_ERR_INVALID_ARG, "N=%lld < 1: no strict prefix", (long long)n_tokens);
    if (interval < 1) return fail(LA_ERR_INVALID_ARG, "C=%lld < 1", (long long)interval);
    if (available_tokens < 0) return fail(LA_ERR_INVALID_ARG, "available=%lld < 0", (long long)available_tokens);
    const int64_t query = (n_tokens - 1) / interval * interval;      // exclude the last prompt token
    const int64_t avail = available_tokens / interval * interval;    // only whole cached blocks
    *boundary_out = std::min(query, avail);
    return LA_OK;
}

la_status la_hybrid_boundary(int64_t n_tokens, int64_t interval, int64_t kv_block_tokens, int64_t kv_cached_tokens,
                             int64_t state_cached_tokens, int64_t *boundary_out, int64_t *kv_blocks_out) {
    if (!boundary_out || !kv_blocks_out) return fail(LA_ERR_INVALID_ARG, "boundary_out and kv_blocks_out are required");
    if (kv_block_tokens < 1) return fail(LA_ERR_INVALID_ARG, "kv_block_tokens=%lld < 1", (long long)kv_block_tokens);
    if (kv_cached_tokens < 0 || state_cached_tokens < 0)
        return fail(LA_ERR_INVALID_ARG, "cached lengths must be >= 0");
    if (interval >= 1 && interval % kv_block_tokens != 0)
        return fail(LA_ERR_MISALIGNED_STATE, "KV blocks of %lld tokens do not tile the checkpoint interval C=%lld",
                    (long long)kv_block_tokens, (long long)interval);
    int64_t b = 0;
    if (la_status e = strict_prefix_boundary(n_tokens, interval, std::min(kv_cached_tokens, state_cached_tokens), &b))
        return e;
    *boundary_out = b;
    *kv_blocks_out = b / kv_block_tokens;
    return LA_OK;
}

la_status la_hybrid_restore(const la_kv_blocks *kv, int32_t n_seqs, int32_t n_heads, int64_t page_elems,
                            const int64_t *boundary_dev, const int64_t *boundary_host, const float *state_pool,
                            int64_t n_state_pages, const int32_t *state_page_ids_dev, float *states,
                            int32_t *err_count_dev, void *stream) {
    if (!kv) return fail(LA_ERR_INVALID_ARG, "kv is NULL");
    if (n_seqs < 0 || n_seqs > 65535) return fail(LA_ERR_INVALID_ARG, "n_seqs=%d outside [0, 65535]", n_seqs);
    if (n_heads < 0 || n_heads > 65535) return fail(LA_ERR_INVALID_ARG, "n_heads=%d outside [0, 65535]", n_heads);
    if (kv->block_tokens < 1) return fail(LA_ERR_INVALID_ARG, "block_tokens=%lld < 1", (long long)kv->block_tokens);
    if (kv->block_bytes <= 0 || kv->block_bytes % 16 != 0)
        return fail(LA_ERR_INVALID_ARG, "block_bytes=%lld must be a positive multiple of 16", (long long)kv->block_bytes);
    if (kv->max_blocks < 0 || kv->max_blocks > 0x7fffffff || kv->n_pool_blocks < 0 || kv->n_pool_blocks > 0x7fffffff ||
        kv->n_cache_blocks < 0 || kv->n_cache_blocks > 0x7fffffff)
        return fail(LA_ERR_INVALID_ARG, "block counts outside [0, 2^31)");
    if (n_seqs == 0) return LA_OK;
    if (!boundary_dev || !boundary_host) return fail(LA_ERR_INVALID_ARG, "boundary_dev and boundary_host are required");
    int64_t nb_max = 0;
    for (int i = 0; i < n_seqs; ++i) {
        const int64_t b = boundary_host[i];
        if (b < 0) return fail(LA_ERR_INVALID_ARG, "boundary[%d]=%lld < 0", i, (long long)b);
        if (b % kv->block_tokens != 0)
            return fail(LA_ERR_MISALIGNED_STATE, "boundary[%d]=%lld is not a multiple of the KV block (%lld tokens)", i,
                        (long long)b, (long long)kv->block_tokens);
        if (b / kv->block_tokens > kv->max_blocks)
            return fail(LA_ERR_INVALID_ARG, "boundary[%d] needs %lld blocks, max_blocks=%lld", i,
                        (long long)(b / kv->block_tokens), (long long)kv->max_blocks);
        nb_max = std::max(nb_max, b / kv->block_tokens);
    }
    if (nb_max + n_heads > 0x7fffffff) return fail(LA_ERR_INVALID_ARG, "too many blocks for one launch");
    const void *kv_pool = nullptr;
    if (nb_max > 0) {
        if (!kv->cache || !kv->src_ids || !kv->dst_ids)
            return fail(LA_ERR_INVALID_ARG, "kv cache, src_ids and dst_ids are required");
        if (!aligned16(kv->cache)) return fail(LA_ERR_INVALID_ARG, "kv cache must be 16-byte aligned");
        if (kv->n_pool_blocks > 0) {
            if (la_status e = resolve_pool(kv->pool, (size_t)kv->n_pool_blocks * kv->block_bytes, &kv_pool, "kv pool"))
                return e;
            if (!aligned16(kv_pool)) return fail(LA_ERR_INVALID_ARG, "kv pool must be 16-byte aligned");
        }
    }
    const void *st_pool = nullptr;
    if (n_heads > 0) {
        if (page_elems <= 0 || page_elems % 4 != 0)
            return fail(LA_ERR_INVALID_ARG, "page_elems=%lld must be a positive multiple of 4", (long long)page_elems);
        if (n_state_pages < 0 || n_state_pages > 0x7fffffff)
            return fail(LA_ERR_INVALID_ARG, "n_state_pages=%lld", (long long)n_state_pages);
        if (!state_page_ids_dev || !states) return fail(LA_ERR_INVALID_ARG, "state_page_ids and states are required");
        if (!aligned16(states)) return fail(LA_ERR_INVALID_ARG, "states must be 16-byte aligned");
        if (n_state_pages > 0) {
            if (la_status e = resolve_pool(state_pool, (size_t)n_state_pages * page_elems * sizeof(float), &st_pool,
                                           "state pool"))
                return e;
            if (!aligned16(st_pool)) return fail(LA_ERR_INVALID_ARG, "state pool must be 16-byte aligned");
        }
    }
    if (nb_max + n_heads == 0) return LA_OK;
    la::HybridArgs a{};
    a.kv_pool = (const la::f32x4 *)kv_pool;
    a.cache = (la::f32x4 *)kv->cache;
    a.src_ids = kv->src_ids;
    a.dst_ids = kv->dst_ids;
    a.boundary = boundary_dev;
    a.state_pool = (const la::f32x4 *)st_pool;
    a.state_ids = state_page_ids_dev;
    a.states = (la::f32x4 *)states;
    a.err = err_count_dev;
    a.kv_vec = kv->block_bytes / 16;
    a.n_pool_blocks = kv->n_pool_blocks;
    a.n_cache_blocks = kv->n_cache_blocks;
    a.max_blocks = kv->max_blocks;
    a.block_tokens = kv->block_tokens;
    a.page_vec = n_heads > 0 ? page_elems / 4 : 0;
    a.n_state_pages = n_heads > 0 ? n_state_pages : 0;
    a.n_heads = n_heads;
    a.nb_max = (int32_t)nb_max;
    const int64_t parts = (std::max(nb_max > 0 ? a.kv_vec : 0, a.page_vec) + la::kHybridPartVec - 1) /
                          la::kHybridPartVec;
    if (parts > 65535) return fail(LA_ERR_INVALID_ARG, "blocks or pages too large for one launch");
    (void)hipGetLastError();
    hipLaunchKernelGGL(la::hybrid_restore_kernel, dim3((unsigned)(nb_max + n_heads), (unsigned)n_seqs, (unsigned)parts),
                       dim3(la::kPageThreads), 0, (hipStream_t)stream, a);
    return hip_check("hybrid restore launch");
}

size_t la_prefill_workspace_bytes(const la_shape *shape, int64_t total_tokens) {
    if (check_shape(shape) != LA_OK || total_tokens < 0) return 0;
    return plan_workspace(shape, total_tokens).total;
}

la_status la_prefill(const la_shape *shape, const void *q, const void *k, const void *v, const float *g,
                     const float *beta, const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host, void *o,
                     float *final_state, float *ckpt_out, const int32_t *ckpt_offsets_dev,
                     const int32_t *ckpt_offsets_host, void *workspace, size_t ws_bytes, void *stream) {
    PrefillCall c{shape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host, nullptr, nullptr, nullptr,
                  o, final_state, ckpt_out, ckpt_offsets_dev, ckpt_offsets_host, workspace, ws_bytes,
                  (hipStream_t)stream};
    return run_prefill(c);
}

la_status la_prefill_resume(const la_shape *shape, const void *q, const void *k, const void *v, const float *g,
                            const float *beta, const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                            const int64_t *start_pos_dev, const int64_t *start_pos_host, const float *state_in,
                            void *o, float *final_state, float *ckpt_out, const int32_t *ckpt_offsets_dev,
                            const int32_t *ckpt_offsets_host, void *workspace, size_t ws_bytes, void *stream) {
    if (!start_pos_dev || !start_pos_host)
        return fail(LA_ERR_INVALID_ARG, "start_pos_dev and start_pos_host are required");
    PrefillCall c{shape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host, start_pos_dev, start_pos_host,
                  state_in, o, final_state, ckpt_out, ckpt_offsets_dev, ckpt_offsets_host, workspace, ws_bytes,
                  (hipStream_t)stream};
    return run_prefill(c);
}

la_status la_prefill_stages(const la_shape *shape, uint32_t stages, const void *q, const void *k, const void *v,
                            const float *g, const float *beta, const int32_t *cu_seqlens_dev,
                            const int32_t *cu_seqlens_host, const int64_t *start_pos_dev,
                            const int64_t *start_pos_host, const float *state_in, void *o, float *final_state,
                            float *ckpt_out, const int32_t *ckpt_offsets_dev, const int32_t *ckpt_offsets_host,
                            void *workspace, size_t ws_bytes, void *stream) {
    if ((start_pos_dev == nullptr) != (start_pos_host == nullptr))
        return fail(LA_ERR_INVALID_ARG, "start_pos_dev and start_pos_host go together");
    PrefillCall c{shape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host, start_pos_dev, start_pos_host,
                  state_in, o, final_state, ckpt_out, ckpt_offsets_dev, ckpt_offsets_host, workspace, ws_bytes,
                  (hipStream_t)stream, stages};
    return run_prefill(c);
}

la_status la_prefill_paged(const la_shape *shape, const la_pages *pages, const void *q, const void *k, const void *v,
                           const float *g, const float *beta, const int32_t *cu_seqlens_dev,
                           const int32_t *cu_seqlens_host, const int64_t *start_pos_dev,
                           const int64_t *start_pos_host, void *o, float *final_state,
                           const int32_t *ckpt_offsets_dev, const int32_t *ckpt_offsets_host, void *workspace,
                           size_t ws_bytes, void *stream) {
    if (!pages) return fail(LA_ERR_INVALID_ARG, "pages is NULL");
    if ((start_pos_dev == nullptr) != (start_pos_host == nullptr))
        return fail(LA_ERR_INVALID_ARG, "start_pos_dev and start_pos_host go together");
    PrefillCall c{shape, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host, start_pos_dev, start_pos_host,
                  nullptr, o, final_state, nullptr, ckpt_offsets_dev, ckpt_offsets_host, workspace, ws_bytes,
                  (hipStream_t)stream, LA_STAGE_ALL, pages};
    return run_prefill(c);
}

la_status la_decode_step(const la_shape *shape, const void *q, const void *k, const void *v, const float *g,
                         const float *beta, float *state, void *o, void *stream) {
    if (la_status e = check_shape(shape)) return e;
    if (!q || !k || !v || !g || !beta || !state || !o)
        return fail(LA_ERR_INVALID_ARG, "q, k, v, g, beta, state and o are required");
    if (!aligned16(state)) return fail(LA_ERR_INVALID_ARG, "state must be 16-byte aligned");
    const size_t io = io_size(shape->io_dtype);
    if ((uintptr_t)q % io || (uintptr_t)k % io || (uintptr_t)v % io || (uintptr_t)o % io)
        return fail(LA_ERR_INVALID_ARG, "q, k, v and o must be aligned to their element size");
    la::DecodeArgs a{q, k, v, g, beta, state, o, shape->n_seqs, shape->n_heads, shape->variant, shape->scale};
    (void)hipGetLastError();
    if (shape->io_dtype == LA_BF16) return decode_dims<__bf16>(shape, a, (hipStream_t)stream);
    return decode_dims<float>(shape, a, (hipStream_t)stream);
}

la_status la_state_save_paged(const float *states, int64_t n_items, int64_t page_elems, float *pool,
                              int64_t n_pages, const int32_t *page_ids_dev, int32_t *err_count_dev, void *stream) {
    if (la_status e = check_paged(states, pool, n_items, page_elems, n_pages, page_ids_dev)) return e;
    if (n_items == 0) return LA_OK;
    (void)hipGetLastError();
    hipLaunchKernelGGL(la::page_save_kernel, dim3((unsigned)n_items), dim3(la::kPageThreads), 0,
                       (hipStream_t)stream, (const la::f32x4 *)states, page_elems / 4, (la::f32x4 *)pool,
                       n_pages, page_ids_dev, err_count_dev);
    return hip_check("page save launch");
}

la_status la_state_restore_paged(const float *pool, int64_t n_pages, const int32_t *page_ids_dev, float *states,
                                 int64_t n_items, int64_t page_elems, int32_t *err_count_dev, void *stream) {
    if (la_status e = check_paged(states, pool, n_items, page_elems, n_pages, page_ids_dev)) return e;
    if (n_items == 0) return LA_OK;
    (void)hipGetLastError();
    hipLaunchKernelGGL(la::page_restore_kernel, dim3((unsigned)n_items), dim3(la::kPageThreads), 0,
                       (hipStream_t)stream, (const la::f32x4 *)pool, n_pages, page_ids_dev, (la::f32x4 *)states,
                       page_elems / 4, err_count_dev);
    return hip_check("page restore launch");
}

la_status la_state_save_host(const float *states, int64_t n_items, int64_t page_elems, float *host_pool,
                             int64_t n_pages, const int32_t *page_ids_dev, int32_t *err_count_dev, void *stream,
                             void *done_event) {
    if (la_status e = check_paged(states, host_pool, n_items, page_elems, n_pages, page_ids_dev)) return e;
    if (n_items == 0) return record_done(done_event, stream);
    float *dev = nullptr;
    if (la_status e = host_pool_device_ptr(host_pool, (size_t)n_pages * page_elems * sizeof(float), &dev)) return e;
    if (!aligned16(dev)) return fail(LA_ERR_INVALID_ARG, "host pool must be 16-byte aligned");
    (void)hipGetLastError();
    hipLaunchKernelGGL(la::page_save_kernel, dim3((unsigned)n_items), dim3(la::kPageThreads), 0,
                       (hipStream_t)stream, (const la::f32x4 *)states, page_elems / 4, (la::f32x4 *)dev,
                       n_pages, page_ids_dev, err_count_dev);
    if (la_status e = hip_check("host-tier save launch")) return e;
    return record_done(done_event, stream);
}

la_status la_state_restore_host(const float *host_pool, int64_t n_pages, const int32_t *page_ids_dev, float *states,
                                int64_t n_items, int64_t page_elems, int32_t *err_count_dev, void *stream,
                                void *done_event) {
    if (la_status e = check_paged(states, host_pool, n_items, page_elems, n_pages, page_ids_dev)) return e;
    if (n_items == 0) return record_done(done_event, stream);
    float *dev = nullptr;
    if (la_status e = host_pool_device_ptr(host_pool, (size_t)n_pages * page_elems * sizeof(float), &dev)) return e;
    if (!aligned16(dev)) return fail(LA_ERR_INVALID_ARG, "host pool must be 16-byte aligned");
    (void)hipGetLastError();
    hipLaunchKernelGGL(la::page_restore_kernel, dim3((unsigned)n_items), dim3(la::kPageThreads), 0,
                       (hipStream_t)stream, (const la::f32x4 *)dev, n_pages, page_ids_dev, (la::f32x4 *)states,
                       page_elems / 4, err_count_dev);
    if (la_status e = hip_check("host-tier restore launch")) return e;
    return record_done(done_event, stream);
}

const char *la_status_string(la_status status) {
    switch (status) {
        case LA_OK: return "LA_OK";
        case LA_ERR_INVALID_ARG: return "LA_ERR_INVALID_ARG";
        case LA_ERR_UNSUPPORTED: return "LA_ERR_UNSUPPORTED";
        case LA_ERR_EMPTY_SUFFIX: return "LA_ERR_EMPTY_SUFFIX";
        case LA_ERR_MISALIGNED_STATE: return "LA_ERR_MISALIGNED_STATE";
        case LA_ERR_HIP: return "LA_ERR_HIP";
        case LA_ERR_WORKSPACE: return "LA_ERR_WORKSPACE";
    }
    return "LA_ERR_UNKNOWN";
}

const char *la_last_error_message(void) { return g_msg; }

void la_trace_set_events(void *const *events, int32_t n_events) {
    if (!events || n_events < 4) {
        g_trace_n = 0;
        return;
    }
    for (int i = 0; i < 4; ++i) g_trace[i] = events[i];
    g_trace_n = 4;
}

}  // extern "C"

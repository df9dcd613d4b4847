// C ABI of the strict-prefix linear-attention prefill library (gfx950).
// Host side: argument validation, the chunk plan's sizes, workspace carving
// and launches.  Kernels live in the headers included below.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <functional>
#include <mutex>
#include <type_traits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "linattn.h"
#include "la_common.h"
#include "gdr_prep.h"
#include "gdr_scan.h"
#include "gdr_out.h"
#include "gdr_xscan.h"
#include "gdr_decode.h"
#include "paged.h"
#include "hybrid.h"

// Workspace of la_prefill_paged_noalloc, for callers that cannot allocate:
// a file-scope device array, one copy per device the library runs on, held
// until the process ends.  Host code reaches it only through the address
// hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

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

// Device address of `scratch` on the current device: looked up once per
// device (with that device current), then reused.  std::call_once makes the
// lookup race-free; the table is written only inside it.
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void *g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

la_status scratch_address(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(LA_ERR_HIP, "no current device for the static scratch (device %d)", dev);
    std::call_once(g_scratch_once[dev], [dev]() {
        void *ptr = nullptr;
        g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = ptr;
    });
    if (g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev])
        return fail(LA_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                    hipGetErrorString(g_scratch_err[dev]));
    *out = g_scratch_ptr[dev];
    return LA_OK;
}

constexpr size_t kRegionAlign = 256;
constexpr int64_t kDeviceCUs = 256;   // compute units of an MI355X (gfx950)

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

size_t io_size(int32_t dtype) { return dtype == LA_BF16 ? 2 : 4; }

// Chunks per segment of the two-level scan (1 = single-level).  A segment
// must divide a checkpoint interval's chunks, so every checkpoint position is
// a segment boundary and a resume from a checkpoint sees the same segments
// (and computes bit-identical states) as the run that wrote it; for the same
// reason the choice depends on the interval only, never on the lengths.  The
// largest such divisor up to 16 balances the two parallel levels against the
// sequential combine.  Intervals of fewer than 8 chunks keep the
// single-level scan: there a segment's map costs more than the chunks it
// replaces.  bf16 operands only.
int seg_chunks(const la_shape *s) {
    if (s->io_dtype != LA_BF16) return 1;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    if (cps < 8) return 1;
    for (int m = std::min(cps, 16); m >= 2; --m)
        if (cps % m == 0) return m;
    return 1;
}

// The kernels a prefill call runs, a function of its shape alone (so a
// resume and the run that wrote its checkpoint always take the same form):
//   bf16: the preparation, then the fused scan (single-level), or the
//         segment maps, the combine and the fused replay (two-level);
//   fp32: the per-chunk preparation, then the one-tile scan with its output
//         wave (dk = 64), or the dk-split scan and the output kernel (dk = 128,
//         whose one-tile state does not fit the register file).
la_form prefill_form(const la_shape *s) {
    if (s->io_dtype == LA_BF16) return seg_chunks(s) > 1 ? LA_FORM_FUSED_TWO_LEVEL : LA_FORM_FUSED_SCAN;
    return s->dk == 128 ? LA_FORM_SPLIT_DK_SCAN : LA_FORM_TILE_SCAN_OUT;
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

// Workspace regions (byte offsets; 0 = absent).  Per chunk slot and head:
//   bf16: the X fragments (6 KB) and the gate block (1 KB), in one block;
//   fp32: -W, K~^T, U~, G, P and Q in operand order, plus the state entering
//         each chunk and U for the output kernel of the dk-split scan.
// The two-level scan adds, per segment slot and head, Phi' (io type), R, D
// and the state entering the segment.
struct WsPlan {
    size_t misc;                             // bf16 forms
    size_t w, kt, ut, g, sc, u, pm, qf;      // fp32 forms
    size_t phi, segr, segd, segst;           // two-level scan (seg_m >= 2)
    int seg_m;
    size_t total;
};

WsPlan plan_workspace(const la_shape *s, int64_t total_tokens) {
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    const int64_t slots = la::total_slots(total_tokens, s->n_seqs, s->ckpt_interval, cps);
    const size_t sh = (size_t)slots * s->n_heads;
    const size_t io = io_size(s->io_dtype);
    const la_form form = prefill_form(s);
    WsPlan p{};
    size_t off = kRegionAlign;   // offset 0 marks an absent region
    auto take = [&](size_t bytes) { const size_t at = off; off = round_up(off + bytes, kRegionAlign); return at; };
    if (s->io_dtype == LA_BF16) {
        p.misc = take(sh * la::kMiscVec * 16);
    } else {
        p.w = take(sh * la::kChunk * s->dk * io);
        p.kt = take(sh * s->dk * la::kChunk * io);
        p.ut = take(sh * la::kChunk * s->dv * io);
        p.g = take(sh * la::kChunk * sizeof(float));
        p.pm = take(sh * la::kChunk * la::kChunk * io);
        p.qf = take(sh * la::kChunk * s->dk * io);
        if (form == LA_FORM_SPLIT_DK_SCAN) {
            p.sc = take(sh * (size_t)s->dk * s->dv * io);
            p.u = take(sh * la::kChunk * s->dv * io);
        }
    }
    p.seg_m = seg_chunks(s);
    if (p.seg_m > 1) {
        const int64_t seg_slots = la::total_slots(total_tokens, s->n_seqs, s->ckpt_interval * (int64_t)p.seg_m, cps);
        const size_t ssh = (size_t)seg_slots * s->n_heads;
        p.phi = take(ssh * s->dk * s->dk * io);
        p.segr = take(ssh * s->dk * s->dv * sizeof(float));
        p.segd = take(ssh * sizeof(float));
        p.segst = take(ssh * s->dk * s->dv * sizeof(float));
    }
    p.total = off;
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
    const la_pages *pages = nullptr;         // paged checkpoints / starting states
};

// Profiling hook (la_trace_set_events): events recorded on the launch stream
// at the start, after the preparation, after the segment maps and combine
// (two-level forms only; at the same point as the previous event otherwise)
// and at the end.
void trace_mark(int i, hipStream_t stream) {
    if (g_trace_n >= 4) (void)hipEventRecord((hipEvent_t)g_trace[i], stream);
}

// Ranks the (sequence, head) chains for dispatch, longest first (equal
// lengths keep sequence order), so the long chains start first.  Batches of
// more than kChainOrderMax chains, or of one sequence, keep the natural
// order.
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

la::ScanArgs scan_args(const PrefillCall &c, const la::Workspace &ws) {
    const la_shape *s = c.shape;
    la::ScanArgs sa{};
    sa.cu = c.cu_dev;
    sa.state_in = c.state_in;
    sa.final_state = c.final_state;
    sa.ckpt = c.ckpt_out;
    sa.ckpt_off = c.ckpt_off_dev;
    sa.n_seqs = s->n_seqs;
    sa.n_heads = s->n_heads;
    sa.C = s->ckpt_interval;
    sa.cps = la::chunks_per_interval(s->ckpt_interval);
    sa.ws = ws;
    sa.seg_m = 1;
    sa.max_seg = 1;
    sa.q = c.q;
    sa.k = c.k;
    sa.v = c.v;
    sa.o = c.o;
    sa.scale = s->scale;
    if (c.pages) {
        sa.pg.pool = c.pages->pool;
        sa.pg.ckpt_ids = c.pages->ckpt_page_ids;
        sa.pg.state_ids = c.pages->state_page_ids;
        sa.pg.err = c.pages->err_count;
        sa.pg.n_pages = (int32_t)c.pages->n_pages;
    }
    order_chains(c, sa.order);
    return sa;
}

// Per-chunk step of one fused-scan workgroup by column width, relative to
// the 64-column form's (measured on the MI355X at dk = dv = 128, all CUs
// busy): narrower workgroups give each wave fewer columns, so a chunk takes
// less time, but a chain then needs more workgroups.
constexpr double kStep32 = 0.87, kStep64 = 1.0;

// Widths of the single-level fused scan for a bf16 call with these
// sequence lengths (cu_host valid).  At dk = dv = 128: 128 columns when the
// chains give every CU two workgroups; else the n_narrow longest chains (a
// multiple of 8, or all) take 32-column workgroups and the others 64, with
// n_narrow minimising an estimate of the scan's span: the longest narrow
// chain, the longest wide chain, or all chunk steps spread over the CUs,
// whichever is longest (a narrow chain runs four workgroups at kStep32 per
// chunk, a wide one two at kStep64).  Other head sizes take 64 columns.
// The widths never change a result.
struct ScanWidths {
    int cw;             // 32, 64 or 128; 0 for a mix of 32 (the first n_narrow ranked chains) and 64
    int64_t n_narrow;
};
ScanWidths fused_scan_widths(const la_shape *s, const int32_t *cu_host) {
    const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
    if (s->dk != 128 || s->dv != 128) return {64, 0};
    if (pairs >= 2 * kDeviceCUs) return {128, 0};
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    int64_t nch[2 * kDeviceCUs];
    double total = 0.0;
    for (int64_t k = 0; k < pairs; ++k) {
        const int i = (int)(k / s->n_heads);
        nch[k] = la::n_chunks((int64_t)cu_host[i + 1] - cu_host[i], s->ckpt_interval, cps);
        total += (double)nch[k];
    }
    // ranked as the dispatch ranks them (longest first; mixing needs that ranking)
    std::sort(nch, nch + pairs, std::greater<int64_t>());
    const bool can_mix = s->n_seqs >= 2 && pairs <= la::kChainOrderMax;
    double narrow_sum = 0.0, best = 0.0;
    int64_t best_k = 0, done = 0;
    auto consider = [&](int64_t k) {
        for (; done < k; ++done) narrow_sum += (double)nch[done];
        const double span = std::max({k > 0 ? kStep32 * (double)nch[0] : 0.0,
                                      k < pairs ? kStep64 * (double)nch[k] : 0.0,
                                      (4.0 * kStep32 * narrow_sum + 2.0 * kStep64 * (total - narrow_sum)) /
                                          (double)kDeviceCUs});
        if (k == 0 || span < best) {
            best = span;
            best_k = k;
        }
    };
    consider(0);
    if (can_mix)
        for (int64_t k = 8; k < pairs; k += 8) consider(k);
    consider(pairs);
    if (best_k == 0) return {64, 0};
    if (best_k == pairs) return {32, pairs};
    return {0, best_k};
}

// Column width of the two-level passes over `units` (sequence, head,
// segment) units: 128 while that still gives every CU two workgroups (dk =
// dv = 128), else 64, which spreads each unit over more CUs.
template <int DK, int DV, int MODE> int two_level_width(int64_t units) {
    constexpr int NCOLS = MODE == la::kXMap ? DK + DV : DV;
    return (DK == 128 && DV == 128 && units * (NCOLS / 128) >= 2 * kDeviceCUs) ? 128 : 64;
}

// The fused scan kernel of one mode over `units` independent units at
// column width cw (32 for the single-level scan only; 128 at dk = dv = 128
// only).  Every column's arithmetic is the same at all widths.
template <int DK, int DV, int MODE>
la_status launch_xscan(const la::ScanArgs &sa, int64_t units, hipStream_t stream, const char *what, int cw) {
    constexpr int NCOLS = MODE == la::kXMap ? DK + DV : DV;
    auto go = [&](auto width) {
        constexpr int CW = decltype(width)::value;
        const int64_t blocks = 8 * (NCOLS / CW) * ((units + 7) / 8);
        hipLaunchKernelGGL((la::gdr_xscan_kernel<DK, DV, MODE, CW>), dim3((unsigned)blocks),
                           dim3(la::xscan_threads(CW, MODE)), 0, stream, sa);
        return hip_check(what);
    };
    if constexpr (DK == 128 && DV == 128) {
        if constexpr (MODE == la::kXScan) {
            if (cw == 32) return go(std::integral_constant<int, 32>{});
        }
        if (cw == 128) return go(std::integral_constant<int, 128>{});
    }
    return go(std::integral_constant<int, 64>{});
}

// bf16: preparation, then the fused scan, or the two-level scan (segment
// maps, combine, fused replay).
template <int DK, int DV>
la_status launch_fused(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    const la_shape *s = c.shape;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    char *base = (char *)c.workspace;
    la::Workspace ws{};
    ws.misc = (uint4 *)(base + p.misc);
    trace_mark(0, c.stream);
    (void)hipGetLastError();
    if (max_chunks > 0) {
        la::XPrepArgs pa{c.k, c.g, c.beta, c.cu_dev, s->n_seqs, s->n_heads, s->ckpt_interval, cps, s->variant,
                         (int32_t)max_chunks, ws.misc,
                         la::chunk_major_map(s->n_seqs, s->n_heads, max_chunks) ? 1 : 0};
        const int64_t blocks = la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks);
        hipLaunchKernelGGL((la::gdr_xprep_kernel<DK>), dim3((unsigned)blocks), dim3(256), 0, c.stream, pa);
        if (la_status e = hip_check("chunk preparation launch")) return e;
    }
    trace_mark(1, c.stream);
    la::ScanArgs sa = scan_args(c, ws);
    const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
    if (p.seg_m > 1) {
        sa.seg_m = p.seg_m;
        sa.max_seg = (int32_t)((max_chunks + p.seg_m - 1) / p.seg_m);
        sa.seg.phi = base + p.phi;
        sa.seg.r = (float *)(base + p.segr);
        sa.seg.d = (float *)(base + p.segd);
        sa.seg.state = (float *)(base + p.segst);
        const int64_t units = pairs * sa.max_seg;
        if (units > 0)
            if (la_status e = launch_xscan<DK, DV, la::kXMap>(sa, units, c.stream, "segment map launch",
                                                              two_level_width<DK, DV, la::kXMap>(units)))
                return e;
        hipLaunchKernelGGL((la::gdr_xcombine_kernel<DK, DV>), dim3((unsigned)(8 * (DV / 16) * ((pairs + 7) / 8))),
                           dim3(64 * (DK / 32)), 0, c.stream, sa);
        if (la_status e = hip_check("segment combine launch")) return e;
        trace_mark(2, c.stream);
        if (units > 0)
            if (la_status e = launch_xscan<DK, DV, la::kXReplay>(sa, units, c.stream, "segment replay launch",
                                                                 two_level_width<DK, DV, la::kXReplay>(units)))
                return e;
    } else {
        trace_mark(2, c.stream);
        const ScanWidths sw = fused_scan_widths(s, c.cu_host);
        if (sw.cw != 0) {
            if (la_status e = launch_xscan<DK, DV, la::kXScan>(sa, pairs, c.stream, "fused scan launch", sw.cw))
                return e;
        } else if constexpr (DK == 128 && DV == 128) {
            sa.n_narrow = (int32_t)sw.n_narrow;
            const int64_t blocks = 4 * sw.n_narrow + 16 * ((pairs - sw.n_narrow + 7) / 8);
            hipLaunchKernelGGL((la::gdr_xscan_mixed_kernel<DK, DV>), dim3((unsigned)blocks), dim3(384), 0, c.stream, sa);
            if (la_status e = hip_check("fused scan launch")) return e;
        }
    }
    trace_mark(3, c.stream);
    return LA_OK;
}

// fp32: per-chunk preparation, then the one-tile scan with its output wave
// (dk = 64), or the dk-split scan and the split output kernel (dk = 128).
template <int DK, int DV>
la_status launch_f32(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    typedef float T;
    const la_shape *s = c.shape;
    const int cps = la::chunks_per_interval(s->ckpt_interval);
    char *base = (char *)c.workspace;
    la::Workspace ws{};
    ws.w = base + p.w;
    ws.kt = base + p.kt;
    ws.ut = base + p.ut;
    ws.g = (float *)(base + p.g);
    ws.sc = p.sc ? base + p.sc : nullptr;
    ws.u = p.u ? base + p.u : nullptr;
    ws.p = base + p.pm;
    ws.qf = base + p.qf;
    const int32_t chunk_major = la::chunk_major_map(s->n_seqs, s->n_heads, max_chunks) ? 1 : 0;
    trace_mark(0, c.stream);
    (void)hipGetLastError();
    if (max_chunks > 0) {
        la::PrepArgs pa{c.q, c.k, c.v, c.g, c.beta, c.cu_dev, s->n_seqs, s->n_heads, s->ckpt_interval, cps,
                        s->variant, (int32_t)max_chunks, ws, chunk_major};
        const int64_t blocks = la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks);
        hipLaunchKernelGGL((la::gdr_prep_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(256), 0, c.stream, pa);
        if (la_status e = hip_check("chunk preparation launch")) return e;
    }
    trace_mark(1, c.stream);
    la::ScanArgs sa = scan_args(c, ws);
    constexpr int NT = DV / 16;
    const int64_t pairs = (int64_t)s->n_seqs * s->n_heads;
    const int64_t blocks = 8 * NT * ((pairs + 7) / 8);
    if constexpr (DK != 128) {   // LA_FORM_TILE_SCAN_OUT (the dk = 128 kernels are not built for it)
        // the scan's output wave produces the output: no output launch
        trace_mark(2, c.stream);
        hipLaunchKernelGGL((la::gdr_scan1o_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(128), 0, c.stream, sa);
        if (la_status e = hip_check("inter-chunk scan launch")) return e;
    } else {
        trace_mark(2, c.stream);
        hipLaunchKernelGGL((la::gdr_scan_kernel<T, DK, DV>), dim3((unsigned)blocks), dim3(64 * la::ScanGeom<DK>::NW), 0,
                           c.stream, sa);
        if (la_status e = hip_check("inter-chunk scan launch")) return e;
        if (max_chunks > 0) {
            la::OutArgs oa{c.o, c.cu_dev, s->n_seqs, s->n_heads, s->ckpt_interval, cps, (int32_t)max_chunks, s->scale,
                           ws, chunk_major};
            const int64_t ob = la::chunk_grid_blocks(s->n_seqs, s->n_heads, max_chunks);
            hipLaunchKernelGGL((la::gdr_out_kernel<T, DK, DV>), dim3((unsigned)ob), dim3(4 * DV), 0, c.stream, oa);
            if (la_status e = hip_check("output launch")) return e;
        }
    }
    trace_mark(3, c.stream);
    return LA_OK;
}

template <int DK, int DV>
la_status launch_prefill(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    if (c.shape->io_dtype == LA_BF16) return launch_fused<DK, DV>(c, p, max_chunks);
    return launch_f32<DK, DV>(c, p, max_chunks);
}

la_status dispatch_dims(const PrefillCall &c, const WsPlan &p, int64_t max_chunks) {
    const int dk = c.shape->dk, dv = c.shape->dv;
    if (dk == 64 && dv == 64) return launch_prefill<64, 64>(c, p, max_chunks);
    if (dk == 64 && dv == 128) return launch_prefill<64, 128>(c, p, max_chunks);
    if (dk == 128 && dv == 64) return launch_prefill<128, 64>(c, p, max_chunks);
    if (dk == 128 && dv == 128) return launch_prefill<128, 128>(c, p, max_chunks);
    return fail(LA_ERR_UNSUPPORTED, "dk=%d dv=%d", dk, dv);
}

la_status run_prefill(const PrefillCall &c) {
    if (la_status e = check_shape(c.shape)) return e;
    const la_shape *s = c.shape;
    const bool resume = c.start_host != nullptr || c.start_dev != nullptr;
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

    return dispatch_dims(c, p, max_chunks);
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

la_form la_prefill_form(const la_shape *shape) {
    if (check_shape(shape) != LA_OK) return LA_FORM_NONE;
    return prefill_form(shape);
}

int la_prefill_scan_columns(const la_shape *shape, const int32_t *cu_seqlens_host, int64_t *narrow_chains_out) {
    if (narrow_chains_out) *narrow_chains_out = 0;
    if (check_shape(shape) != LA_OK || shape->io_dtype != LA_BF16 || !cu_seqlens_host || cu_seqlens_host[0] != 0)
        return 0;
    const int cps = la::chunks_per_interval(shape->ckpt_interval);
    int64_t max_chunks = 0;
    for (int i = 0; i < shape->n_seqs; ++i) {
        const int64_t len = (int64_t)cu_seqlens_host[i + 1] - cu_seqlens_host[i];
        if (len < 0 || cu_seqlens_host[i + 1] < 0) return 0;
        max_chunks = std::max(max_chunks, la::n_chunks(len, shape->ckpt_interval, cps));
    }
    if (prefill_form(shape) == LA_FORM_FUSED_SCAN) {
        const ScanWidths sw = fused_scan_widths(shape, cu_seqlens_host);
        if (narrow_chains_out) *narrow_chains_out = sw.cw == 32 ? (int64_t)shape->n_seqs * shape->n_heads : sw.n_narrow;
        return sw.cw == 0 ? 64 : sw.cw;
    }
    const int64_t units = (int64_t)shape->n_seqs * shape->n_heads * ((max_chunks + seg_chunks(shape) - 1) / seg_chunks(shape));
    return (shape->dk == 128 && shape->dv == 128) ? two_level_width<128, 128, la::kXReplay>(units)
                                                  : two_level_width<64, 64, la::kXReplay>(units);
}

la_status la_checkpoint_rows(int32_t n_seqs, const int32_t *cu_seqlens_host, const int64_t *start_pos_host,
                             int64_t interval, int32_t *offsets_out, int64_t *total_rows_out) {
    if (n_seqs < 0) return fail(LA_ERR_INVALID_ARG, "n_seqs=%d < 0", n_seqs);
    if (interval < 1) return fail(LA_ERR_INVALID_ARG, "C=%lld < 1", (long long)interval);
    if (!total_rows_out || (n_seqs > 0 && (!cu_seqlens_host || !offsets_out)))
        return fail(LA_ERR_INVALID_ARG, "cu_seqlens_host, offsets_out and total_rows_out are required");
    int64_t row = 0;
    for (int i = 0; i < n_seqs; ++i) {
        const int64_t len = (int64_t)cu_seqlens_host[i + 1] - cu_seqlens_host[i];
        const int64_t b = start_pos_host ? start_pos_host[i] : 0;
        if (len < 0) return fail(LA_ERR_INVALID_ARG, "cu_seqlens decreases at sequence %d", i);
        if (b < 0 || b > ((int64_t)1 << 40)) return fail(LA_ERR_INVALID_ARG, "start_pos[%d]=%lld", i, (long long)b);
        if (row > 0x7fffffff) return fail(LA_ERR_INVALID_ARG, "more than 2^31 checkpoint rows");
        offsets_out[i] = (int32_t)row;
        // checkpoints at the absolute multiples of C in (B_i, B_i + len_i]
        row += (b + len) / interval - b / interval;
    }
    if (row > 0x7fffffff) return fail(LA_ERR_INVALID_ARG, "more than 2^31 checkpoint rows");
    *total_rows_out = row;
    return LA_OK;
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
                  (hipStream_t)stream, pages};
    return run_prefill(c);
}

la_status la_prefill_paged_noalloc(const la_shape *shape, const la_pages *pages, const void *q, const void *k,
                                   const void *v, const float *g, const float *beta, const int32_t *cu_seqlens_dev,
                                   const int32_t *cu_seqlens_host, const int64_t *start_pos_dev,
                                   const int64_t *start_pos_host, void *o, float *final_state,
                                   const int32_t *ckpt_offsets_dev, const int32_t *ckpt_offsets_host, void *stream) {
    if (la_status e = check_shape(shape)) return e;
    if (!cu_seqlens_host) return fail(LA_ERR_INVALID_ARG, "cu_seqlens_host is required");
    const int64_t total = cu_seqlens_host[shape->n_seqs];
    if (total < 0) return fail(LA_ERR_INVALID_ARG, "cu_seqlens[n_seqs]=%lld", (long long)total);
    const size_t need = plan_workspace(shape, total).total;
    if (need > kScratchBytes)
        return fail(LA_ERR_WORKSPACE, "the call needs %zu bytes of workspace; the static scratch holds %zu", need,
                    kScratchBytes);
    void *ws = nullptr;
    if (la_status e = scratch_address(&ws)) return e;
    return la_prefill_paged(shape, pages, q, k, v, g, beta, cu_seqlens_dev, cu_seqlens_host, start_pos_dev,
                            start_pos_host, o, final_state, ckpt_offsets_dev, ckpt_offsets_host, ws, kScratchBytes,
                            stream);
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

// Inter-chunk scan: the sequential part of the prefill.
//
// One workgroup owns 16 state columns (a dv tile) of one (sequence, head);
// those columns evolve independently of the others.  Its NW = DK / 32 waves
// split the dk rows of the state: wave w keeps rows [32w, 32w + 32) of the
// fp32 state in MFMA accumulator registers for the whole sequence.  Per
// chunk, with S the state entering it:
//
//   U      = U~ - W S           every wave contracts its own 32 state rows
//                               (one 32-deep MFMA k-step) into a partial
//                               64 x 16 product; the partials meet in LDS,
//                               wave w sums row tile w and adds U~.
//   S_next = exp(G_63) S + K~^T U
//                               every wave updates its own 32 rows from
//                               the whole of U (read back from LDS).
//
// The state enters both products straight from its accumulator layout; the
// -W and K~^T operands were written by the preparation kernel in the
// matching contraction order (perm_row), so a wave's operand slice is a run
// of whole 16-byte vectors.  Operands are prefetched four chunks ahead.  The
// workgroup also hands the output kernel the state entering each chunk and
// U (io type), and writes fp32 checkpoints and the final state.
#pragma once
#include "la_common.h"
#include "gdr_out.h"

namespace la {

// Two-level scan, per segment slot and head (a segment is seg_m consecutive
// chunks of one sequence; seg_m divides the chunks per checkpoint interval,
// so every checkpoint position is a segment boundary).  Over a segment the
// state map is affine: S_out = D S_in + Phi' S_in + R, with D the product of
// the chunk decays, Phi' (dk x dk) the rest of the linear part and R
// (dk x dv) the offset.
struct SegWorkspace {
    void *phi;        // Phi' in the io type, [DK][DK], columns in A-operand order
    float *r;         // R, fp32, C-layout tiles [DV/16][DK/16][64 lanes][4]
    float *d;         // D, fp32, one value per segment slot and head
    float *state;     // state entering the segment, fp32 C-layout tiles (segments >= 1)
};

// Paged state I/O: checkpoints written straight into pool pages and the
// starting state read straight from one (the page save and restore of a
// reload folded into the scan).
struct PageIO {
    float *pool;                  // [n_pages][DK * DV] fp32, or null
    const int32_t *ckpt_ids;      // page of checkpoint row r, head h at [r * H + h] (-1: not written), or null
    const int32_t *state_ids;     // page of the state (sequence i, head h) starts from at [i * H + h]
                                  // (-1: zero state), or null
    int32_t *err;                 // optional: +1 per id outside [-1, n_pages)
    int32_t n_pages;
};

// Dispatch order of the (sequence, head) chains: the chain of rank k is
// pair[k] when n > 0, else pair k.  The host ranks chains by length,
// longest first: workgroups are dealt to XCDs round-robin and, within an
// XCD, to its CUs in dispatch order, so the long chains start first and
// each CU's share of chain-chunks evens out (a scan workgroup's chunk step
// is bound by its CU's memory pipe, which the workgroups on that CU share).
constexpr int kChainOrderMax = 1024;
struct ChainOrder {
    int32_t n;
    uint16_t pair[kChainOrderMax];
};

struct ScanArgs {
    const int32_t *cu;
    const float *state_in;        // [n_seqs, H, DK, DV] or null (zero state)
    float *final_state;           // [n_seqs, H, DK, DV] or null
    float *ckpt;                  // [rows, H, DK, DV] or null
    const int32_t *ckpt_off;      // [n_seqs]
    int32_t n_seqs, n_heads, C, cps;
    Workspace ws;
    int32_t seg_m, max_seg;       // two-level scan only
    SegWorkspace seg;
    void *o;                      // scans with output: output [T, H, dv] (io type)
    float scale;
    const void *q, *k, *v;        // fused scan: the inputs [T, H, dk | dv] (bf16)
    PageIO pg;
    ChainOrder order;
    int32_t n_narrow;             // mixed-width fused scan: chains (ranked) in 32-column workgroups
};

// The chain of workgroup rank k (see ChainOrder); -1 past the last chain.
__device__ inline int chain_of_rank(const ScanArgs &a, int k) {
    if (k >= a.n_seqs * a.n_heads) return -1;
    return a.order.n > 0 ? (int)a.order.pair[k] : k;
}

// Counts an id outside [-1, n_pages) once: count is set in one wave per
// (sequence, head), and one lane adds.
__device__ inline void count_bad_id(const PageIO &pg, int id, bool count) {
    if (count && pg.err && (id < -1 || id >= pg.n_pages) && (threadIdx.x & 63) == 0) atomicAdd(pg.err, 1);
}

// The state (sequence seq, head h) starts from: its rows of state_in, the
// pool page the state page table names, or null for the zero state (no
// state_in; page id -1; a page id out of range, which is counted).
__device__ inline const float *start_state(const ScanArgs &a, int seq, int h, size_t elems, bool count) {
    const size_t item = (size_t)seq * a.n_heads + h;
    if (a.pg.state_ids) {
        const int id = a.pg.state_ids[item];
        count_bad_id(a.pg, id, count);
        return (id >= 0 && id < a.pg.n_pages) ? a.pg.pool + (size_t)id * elems : nullptr;
    }
    return a.state_in ? a.state_in + item * elems : nullptr;
}

// Destinations of the checkpoints of one (sequence, head), in order: rows
// row0, row0 + 1, ... of the dense array, or the pool pages the checkpoint
// page table names for those rows (null: not written).  A page id is read
// with the operands of the chunk (or segment) that ends on its checkpoint,
// load_id(row) in the operand prefetch, so no checkpoint waits on a read.
struct CkptDst {
    float *dense, *pool;
    int32_t *err;
    __amdgpu_buffer_rsrc_t ids;   // this (sequence, head)'s page ids, stride H (no records when dense)
    size_t elems;
    int H, n_pages, n_rows, k;
    bool paged, count;

    __device__ void init(const ScanArgs &a, int seq, int h, int len, size_t E, bool cnt) {
        H = a.n_heads;
        elems = E;
        count = cnt;
        pool = a.pg.pool;
        err = a.pg.err;
        n_pages = a.pg.n_pages;
        n_rows = len / a.C;               // positions are local and start on a multiple of C
        k = 0;
        paged = a.pg.ckpt_ids != nullptr;
        dense = (!paged && a.ckpt) ? a.ckpt + ((size_t)a.ckpt_off[seq] * H + h) * E : nullptr;
        const int32_t *base = paged ? a.pg.ckpt_ids + (size_t)a.ckpt_off[seq] * H + h : a.pg.ckpt_ids;
        // the values are wave-uniform; readfirstlane keeps the resource in
        // scalar registers (a vector-register resource costs a loop per read)
        const uint64_t bp = (uint64_t)base;
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)bp);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(bp >> 32));
        const uint32_t bytes = (uint32_t)__builtin_amdgcn_readfirstlane(paged ? n_rows * H * 4 : 0);
        ids = make_rsrc((const void *)(((uint64_t)hi << 32) | lo), bytes);
    }
    // Issues the read of the page id of local checkpoint row r (uniform; rows
    // past the last read as 0 and are never used).
    __device__ int load_id(int r) const {
        return __builtin_amdgcn_raw_buffer_load_b32(ids, (int)((uint32_t)r * (uint32_t)H * 4u), 0, 0);
    }
    // Page ids of local rows [win, win + 64) in the lanes (lane l: row
    // win + l), read once per 64 rows: a read per checkpoint would put a wait
    // for every store in flight before the next one.
    int idv = 0, win = 0;
    __device__ void load_window(int r0) {
        win = r0;
        const uint32_t lane = threadIdx.x & 63;
        idv = __builtin_amdgcn_raw_buffer_load_b32(ids, (int)(((uint32_t)r0 + lane) * (uint32_t)H * 4u), 0, 0);
        // wait here, once: a wait at the first use inside the loop would also
        // wait for every checkpoint store issued since
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    }
    // Page id of local row r (uniform; rows are visited in increasing order).
    __device__ int window_id(int r) {
        if (r - win >= 64) load_window(r);
        return __builtin_amdgcn_readlane(idv, r - win);
    }
    // Destination of the next checkpoint; id is load_id() or window_id() of its row.
    __device__ float *next(int id) {
        float *d = nullptr;
        if (paged) {
            id = __builtin_amdgcn_readfirstlane(id);
            if (count && err && (id < -1 || id >= n_pages) && (threadIdx.x & 63) == 0) atomicAdd(err, 1);
            if (id >= 0 && id < n_pages) d = pool + (size_t)id * elems;
        } else if (dense) {
            d = dense + (size_t)k * H * elems;
        }
        ++k;
        return d;
    }
};

// Chunk bounds of one sequence, advanced by additions only (the plan of
// chunk_range without a division per chunk).  All counters are 32-bit:
// sequence lengths and C are below 2^31, and 64-bit compares in the loop
// would need vector temporaries that alias in-flight operand loads.
struct ChunkCursor {
    int pos, next_ck, len, C;
    // Moves past the next chunk; true when that chunk ends on a multiple of C.
    __device__ bool advance() {
        const int hi = min(pos + kChunk, min(next_ck, len));
        pos = hi;
        if (hi != next_ck) return false;
        next_ck += C;
        return true;
    }
};

// Writes NTILE 16-row tiles of fp32 state held in C layout (lane: column
// voff's column, rows 4 * (lane / 16) + i of each tile) to a row-major
// [rows, DV] block starting at dst; voff is the lane's byte offset of its
// first row.  Buffer stores with scalar bases keep the store addresses out
// of vector registers.
template <int NTILE, int DV>
__device__ inline void store_state_tiles(float *dst, const f32x4 (&S)[NTILE], uint32_t voff) {
    const auto r = make_rsrc(dst, NTILE * 16 * DV * sizeof(float));
#pragma unroll
    for (int t = 0; t < NTILE; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_int(S[t][i]), r, (int)voff,
                                                  (16 * t + i) * DV * (int)sizeof(float), 0);
}

// State tiles in C layout ([tile][row tile][lane] of f32x4): the two-level
// scan's segment-entering states, written by the combine and read by the
// replay (one 16-byte access per row tile and lane).
template <int RT>
__device__ inline void store_state_c(float *base, int tile, const f32x4 (&S)[RT]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int t = 0; t < RT; ++t)
        ((float4 *)base)[(tile * RT + t) * 64 + lane] = make_float4(S[t][0], S[t][1], S[t][2], S[t][3]);
}

template <int RT>
__device__ inline void load_state_c(const float *base, int tile, f32x4 (&S)[RT]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
        const float4 v = ((const float4 *)base)[(tile * RT + t) * 64 + lane];
        S[t] = f32x4{v.x, v.y, v.z, v.w};
    }
}

constexpr int kScanPrefetch = 4;   // chunks of operands in flight ahead of the one computed

// Runs step(chunk) over chunks 0 .. nch-1 with the operands of the next PF
// chunks in flight, in a ring of PF + 1 operand sets.  The main loop is
// unrolled over the ring so every ring index is a compile-time constant and
// its body has no branch; a prefetch past the last chunk re-reads the last
// one.  The final nch mod (PF + 1) chunks were prefetched by the main loop.
template <int PF, typename Ops, typename Load, typename Step>
__device__ inline void scan_ring(int nch, Load &load, Step &step, Ops *) {
    constexpr int NB = PF + 1;
    if (nch <= 0) return;
    Ops ops[NB];
#pragma unroll
    for (int u = 0; u < PF; ++u) load(ops[u], min(u, nch - 1));
    int j = 0;
    for (; j + NB <= nch; j += NB) {
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            load(ops[(u + PF) % NB], min(j + u + PF, nch - 1));
            step(ops[u], j + u);
        }
    }
#pragma unroll
    for (int u = 0; u < NB - 1; ++u)
        if (j + u < nch) step(ops[u], j + u);
}

template <int DK> struct ScanGeom {
    static constexpr int NW = DK / 32;      // waves per workgroup (32 state rows each)
    static constexpr int MTW = 4 / NW;      // U row tiles each wave reduces
};

template <typename T, int DK, int DV>
__global__ __launch_bounds__(64 * (DK / 32)) void gdr_scan_kernel(ScanArgs a) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    constexpr int KW = M::KW, VEC = Vec<T>::N;
    constexpr int NW = ScanGeom<DK>::NW, MTW = ScanGeom<DK>::MTW;
    constexpr int NT = DV / 16;             // workgroups per (sequence, head)
    constexpr int FS = DK / 4;              // per-lane operand values over dk (all waves)
    constexpr int FU = kChunk / 4;          // per-lane operand values over chunk rows
    constexpr int FW = 8;                   // per-lane values of one wave's 32-row dk slice
    constexpr int VW = FW / VEC;            // 16-byte vectors per slice
    constexpr int VU = FU / VEC;
    static_assert(FW % VEC == 0 && FU % VEC == 0 && NW * 32 == DK, "tiling");

    __shared__ f32x4 part[NW][4][64];       // partial products W_w S_w, C-layout
    __shared__ uint4 ubuf[VU][64];          // U in the io type, B-operand order

    // w is uniform per wave; readfirstlane makes that visible to the compiler
    // so every operand address is a scalar base plus the lane offset.
    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, c16 = lane & 15;
    // XCD-aware mapping: workgroups are dealt to the 8 XCDs round-robin; the
    // NT workgroups of one (sequence, head) land on one XCD and share the
    // chunk operands through its L2.
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = chain_of_rank(a, xcd + 8 * (q / NT)), tile = q % NT;
    const int H = a.n_heads;
    if (pair < 0) return;
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int64_t base = slot_base_dev(cu0, seq, a.C, a.cps);
    const size_t state_off = (size_t)pair * DK * DV;
    const int col = 16 * tile + c16;

    // this wave's state rows: tiles 2w and 2w + 1
    f32x4 S[2];
    const float *src = start_state(a, seq, h, (size_t)DK * DV, tile == 0 && w == 0);
    if (src) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                S[t][i] = src[(size_t)(32 * w + 16 * t + 4 * g16 + i) * DV + col];
    } else {
        S[0] = zero4();
        S[1] = zero4();
    }
    ChunkCursor cur{0, a.C, len, a.C};
    CkptDst ck;
    ck.init(a, seq, h, len, (size_t)DK * DV, tile == 0 && w == 0);
    const uint32_t lane_off = 4u * (uint32_t)(4 * g16 * DV + col);   // C-layout store offset
    // Drain the counters once here: without it the waitcnt pass sees the
    // state loads as possibly pending at the loop header and waits on the
    // in-flight operand prefetch in every iteration.
    __builtin_amdgcn_s_waitcnt(0);

    struct Ops {
        uint4 wn[4][VW];      // -W rows (4 row tiles), this wave's dk slice
        uint4 kt[2][VU];      // K~^T rows of this wave's 2 dk tiles, all chunk rows
        f32x4 ut[MTW];        // U~ row tiles this wave reduces
        float gl;             // G_63
        int ckid;             // page id of the checkpoint this chunk would end (paged)
    };
    const uint32_t lane16 = 16u * (uint32_t)lane;
    auto load = [&](Ops &o, int jj) {
        const int64_t sh = (base + jj) * H + h;
        // issue order: gate, U~, -W, K~^T (earliest-needed last is fine: each
        // use waits only for the loads issued before it)
        o.gl = buf_load4f(make_rsrc(a.ws.g + sh * kChunk, kChunk * sizeof(float)), 0u, 4u * (kChunk - 1));
        o.ckid = ck.load_id(jj / a.cps);
        const auto ru = make_rsrc((const T *)a.ws.ut + sh * L::ut_elems, L::ut_elems * sizeof(T));
#pragma unroll
        for (int m = 0; m < MTW; ++m) o.ut[m] = load_ut<T>(ru, (uint32_t)lane, (uint32_t)(tile * 4 + w * MTW + m));
        const auto rw = make_rsrc((const T *)a.ws.w + sh * L::w_elems, L::w_elems * sizeof(T));
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int v = 0; v < VW; ++v) o.wn[mt][v] = buf_load16(rw, lane16, 1024u * (mt * (FS / VEC) + w * VW + v));
        const auto rk = make_rsrc((const T *)a.ws.kt + sh * L::kt_elems, L::kt_elems * sizeof(T));
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int v = 0; v < VU; ++v) o.kt[t][v] = buf_load16(rk, lane16, 1024u * ((2 * w + t) * VU + v));
    };

    auto step = [&](const Ops &o, int j) {
        const int64_t sh = (base + j) * H + h;
        // state entering the chunk as B operand over this wave's dk slice
        T sb[FW];
#pragma unroll
        for (int f = 0; f < FW; ++f) sb[f] = from_f32<T>(S[f >> 2][f & 3]);
        {
            const auto rs = make_rsrc((T *)a.ws.sc + sh * L::sc_elems, L::sc_elems * sizeof(T));
#pragma unroll
            for (int v = 0; v < VW; ++v)
                buf_store16(*(const uint4 *)&sb[v * VEC], rs, lane16, 1024u * (tile * (FS / VEC) + w * VW + v));
        }
        // partial products over this wave's 32 state rows; the wave that
        // reduces row tile mt starts its partial from U~
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const T *wv = (const T *)&o.wn[mt][0];
            f32x4 acc = zero4();
#pragma unroll
            for (int m = 0; m < MTW; ++m)
                if (mt == w * MTW + m) acc = o.ut[m];
#pragma unroll
            for (int ks = 0; ks < FW / KW; ++ks)
                acc = M::mma(M::pack(&wv[ks * KW]), M::pack(&sb[ks * KW]), acc);
            part[w][mt][lane] = acc;
        }
        __syncthreads();
        // wave w reduces U row tiles [w*MTW, (w+1)*MTW): U = sum of partials
#pragma unroll
        for (int m = 0; m < MTW; ++m) {
            const int mt = w * MTW + m;
            f32x4 pp[NW];
#pragma unroll
            for (int p = 0; p < NW; ++p) pp[p] = part[p][mt][lane];
            f32x4 u = pp[0];
#pragma unroll
            for (int p = 1; p < NW; ++p) u += pp[p];
            // flat B-operand index 4 * mt + i
            T *dst = (T *)&ubuf[(4 * mt) / VEC][lane] + (4 * mt) % VEC;
#pragma unroll
            for (int i = 0; i < 4; ++i) dst[i] = from_f32<T>(u[i]);
        }
        __syncthreads();
        uint4 ub[VU];
#pragma unroll
        for (int v = 0; v < VU; ++v) ub[v] = ubuf[v][lane];
        {
            const auto rs = make_rsrc((T *)a.ws.u + sh * L::u_elems, L::u_elems * sizeof(T));
#pragma unroll
            for (int v = 0; v < VU; ++v)
                if (v % NW == w) buf_store16(ub[v], rs, lane16, 1024u * (tile * VU + v));
        }
        // S = exp(G_63) S + K~^T U on this wave's rows
        const float decay = expf(o.gl);
        const T *uvals = (const T *)&ub[0];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const T *kv = (const T *)&o.kt[t][0];
            f32x4 acc = S[t] * decay;
#pragma unroll
            for (int ks = 0; ks < FU / KW; ++ks)
                acc = M::mma(M::pack(&kv[ks * KW]), M::pack(&uvals[ks * KW]), acc);
            S[t] = acc;
        }
        // checkpoint when the chunk ends on a multiple of C
        if (cur.advance()) {
            if (float *d = ck.next(o.ckid)) store_state_tiles<2, DV>(d + (size_t)32 * w * DV, S, lane_off);
        }
    };

    // Operand ring: chunk j computes while chunks j + 1 .. j + kScanPrefetch
    // are in flight.  Operands come from MALL/HBM (each kernel starts with
    // cold L2s), so several chunks of latency must be covered.
    scan_ring<kScanPrefetch>(nch, load, step, (Ops *)nullptr);

    if (a.final_state) store_state_tiles<2, DV>(a.final_state + state_off + (size_t)32 * w * DV, S, lane_off);
}


// Operand forms of the state entering a chunk and of U, handed from the scan
// wave to the output wave of the same workgroup through LDS: two slots
// (chunk parity), each lane's values as 16-byte vectors [vector][lane].
template <typename T, int DK> struct Handoff {
    static constexpr int VS = DK / 4 / Vec<T>::N, VU = kChunk / 4 / Vec<T>::N;
    uint4 sb[2][VS][64];
    uint4 ub[2][VU][64];
};

// Workgroup barrier that orders LDS only: the release fence waits for this
// wave's LDS accesses (not for its global loads in flight).
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Single-wave form.  One wave owns a 16-column tile of the state and all DK
// rows, kept in fp32 MFMA result registers, so a chunk needs no workgroup
// synchronisation: 4 * DK/32 MFMAs for U = U~ - W S and 2 * DK/16 for the
// state update, with the next chunk's operands in flight while one is
// computed.  scan1_chunks runs the whole sequence of one (sequence, head) on
// one tile and writes the checkpoints.  It hands the state entering each
// chunk and U to the split output kernel through the workspace or, with
// HANDOFF, to the workgroup's output wave through the LDS slots hs (one
// barrier per chunk).  HANDOFF is a compile-time choice: a run-time test
// would split a chunk's step into several basic blocks, and the load/MFMA
// interleave below is scheduled within one block.
template <typename T, int DK, int DV, bool HANDOFF>
__device__ inline void scan1_chunks(const ScanArgs &a, int seq, int h, int tile, int len, int64_t base,
                                    int nch, f32x4 (&S)[DK / 16], Handoff<T, DK> *hs) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    constexpr int KW = M::KW, VEC = Vec<T>::N;
    constexpr int RT = DK / 16;             // state row tiles
    constexpr int FS = DK / 4;              // per-lane operand values over dk
    constexpr int FU = kChunk / 4;          // per-lane operand values over chunk rows
    constexpr int VS = FS / VEC, VU = FU / VEC;
    constexpr int kMfmas = 4 * (FS / KW) + RT * (FU / KW);       // per chunk
    constexpr int kLoads = 1 + 4 + 4 * VS + RT * VU;              // operand loads per chunk

    const int lane = threadIdx.x & 63, g16 = lane >> 4, c16 = lane & 15;
    const int H = a.n_heads;
    ChunkCursor cur{0, a.C, len, a.C};
    CkptDst ck;
    ck.init(a, seq, h, len, (size_t)DK * DV, tile == 0);
    const uint32_t lane_off = 4u * (uint32_t)(4 * g16 * DV + 16 * tile + c16);
    // Drain the counters once here: without it the waitcnt pass sees the
    // state loads as possibly pending at the loop header and waits on the
    // in-flight operand prefetch in every iteration.
    __builtin_amdgcn_s_waitcnt(0);

    struct Ops {
        float gl;
        int ckid;             // page id of the checkpoint this chunk would end (paged)
        f32x4 ut[4];
        uint4 wn[4][VS];
        uint4 kt[RT][VU];
    };
    const uint32_t lane16 = 16u * (uint32_t)lane;
    auto load = [&](Ops &o, int jj) {
        const int64_t sh = (base + jj) * H + h;
        o.gl = buf_load4f(make_rsrc(a.ws.g + sh * kChunk, kChunk * sizeof(float)), 0u, 4u * (kChunk - 1));
        o.ckid = ck.load_id(jj / a.cps);
        const auto ru = make_rsrc((const T *)a.ws.ut + sh * L::ut_elems, L::ut_elems * sizeof(T));
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) o.ut[mt] = load_ut<T>(ru, (uint32_t)lane, (uint32_t)(tile * 4 + mt));
        const auto rw = make_rsrc((const T *)a.ws.w + sh * L::w_elems, L::w_elems * sizeof(T));
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int v = 0; v < VS; ++v) o.wn[mt][v] = buf_load16(rw, lane16 + 1024u * (mt * VS + v), 0u);
        const auto rk = make_rsrc((const T *)a.ws.kt + sh * L::kt_elems, L::kt_elems * sizeof(T));
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int v = 0; v < VU; ++v) o.kt[t][v] = buf_load16(rk, lane16 + 1024u * (t * VU + v), 0u);
    };
    auto step = [&](const Ops &o, int jj) {
        const int64_t sh = (base + jj) * H + h;
        T sb[FS];
#pragma unroll
        for (int f = 0; f < FS; ++f) sb[f] = from_f32<T>(S[f >> 2][f & 3]);
        if constexpr (HANDOFF) {
#pragma unroll
            for (int v = 0; v < VS; ++v) hs->sb[jj & 1][v][lane] = *(const uint4 *)&sb[v * VEC];
        } else {
            const auto rs = make_rsrc((T *)a.ws.sc + sh * L::sc_elems, L::sc_elems * sizeof(T));
#pragma unroll
            for (int v = 0; v < VS; ++v)
                buf_store16(*(const uint4 *)&sb[v * VEC], rs, lane16, 1024u * (tile * VS + v));
        }
        f32x4 U[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const T *wv = (const T *)&o.wn[mt][0];
            f32x4 acc = o.ut[mt];
#pragma unroll
            for (int ks = 0; ks < FS / KW; ++ks)
                acc = M::mma(M::pack(&wv[ks * KW]), M::pack(&sb[ks * KW]), acc);
            U[mt] = acc;
        }
        T ub[FU];
#pragma unroll
        for (int f = 0; f < FU; ++f) ub[f] = from_f32<T>(U[f >> 2][f & 3]);
        if constexpr (HANDOFF) {
#pragma unroll
            for (int v = 0; v < VU; ++v) hs->ub[jj & 1][v][lane] = *(const uint4 *)&ub[v * VEC];
        } else {
            const auto rs = make_rsrc((T *)a.ws.u + sh * L::u_elems, L::u_elems * sizeof(T));
#pragma unroll
            for (int v = 0; v < VU; ++v)
                buf_store16(*(const uint4 *)&ub[v * VEC], rs, lane16, 1024u * (tile * VU + v));
        }
        const float decay = expf(o.gl);
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            const T *kv = (const T *)&o.kt[t][0];
            f32x4 acc = S[t] * decay;
#pragma unroll
            for (int ks = 0; ks < FU / KW; ++ks)
                acc = M::mma(M::pack(&kv[ks * KW]), M::pack(&ub[ks * KW]), acc);
            S[t] = acc;
        }
        // One wave issues both the MFMA chain and the next chunk's operand
        // loads (issued just before this step, in the same scheduling
        // region).  Back to back, the loads stall the in-order issue on the
        // memory pipeline while the matrix core idles; one load per MFMA
        // keeps both busy.
#pragma unroll
        for (int i = 0; i < kMfmas; ++i) {
            if (i < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
        }
        if (kLoads > kMfmas) __builtin_amdgcn_sched_group_barrier(0x020, kLoads - kMfmas, 0);
        if (cur.advance()) {
            if (float *d = ck.next(o.ckid)) store_state_tiles<RT, DV>(d, S, lane_off);
        }
        if constexpr (HANDOFF) lds_barrier();   // this chunk's slot is written; the output wave may read it
    };
    scan_ring<1>(nch, load, step, (Ops *)nullptr);
}

// The output wave of the scan-with-output kernel: per chunk, waits for the
// scan wave's handoff of that chunk, then computes and stores the chunk's
// output for the tile (out_tile).  Its own operands (Q and P fragments, gates) are
// loaded one chunk ahead.  It passes exactly one barrier per chunk, as the
// scan wave does; reading slot j & 1 before the barrier of chunk j + 1 keeps
// the scan wave from overwriting it (that write follows that barrier).
template <typename T, int DK, int DV>
__device__ inline void out_wave_chunks(const ScanArgs &a, int h, int tile, int64_t cu0, int len, int64_t base,
                                       int nch, const Handoff<T, DK> *hs) {
    using F = OutFrag<T, DK>;
    constexpr int VEC = Vec<T>::N, VS = Handoff<T, DK>::VS, VU = Handoff<T, DK>::VU;
    const int lane = threadIdx.x & 63, H = a.n_heads;
    ChunkCursor cur{0, a.C, len, a.C};
    auto load = [&](F &f, int jj) { load_out_frag<T, DK>(f, a.ws, (base + jj) * H + h); };
    auto step = [&](const F &f, int jj) {
        const int lo = cur.pos;
        cur.advance();
        const int n = cur.pos - lo;
        lds_barrier();
        T sb[VS * VEC], ub[VU * VEC];
#pragma unroll
        for (int v = 0; v < VS; ++v) *(uint4 *)&sb[v * VEC] = hs->sb[jj & 1][v][lane];
#pragma unroll
        for (int v = 0; v < VU; ++v) *(uint4 *)&ub[v * VEC] = hs->ub[jj & 1][v][lane];
        out_tile<T, DK>(f, sb, ub, a.scale, (T *)a.o + ((cu0 + lo) * H + h) * DV, n, H, DV, tile);
    };
    scan_ring<1>(nch, load, step, (F *)nullptr);
}

// Loads a [DK][DV] fp32 state's tile into C layout (or zeros for null).
template <int DK, int DV>
__device__ inline void load_state_tile(const float *src, int tile, f32x4 (&S)[DK / 16]) {
    const int lane = threadIdx.x & 63, g16 = lane >> 4, col = 16 * tile + (lane & 15);
    if (src) {
#pragma unroll
        for (int t = 0; t < DK / 16; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) S[t][i] = src[(size_t)(16 * t + 4 * g16 + i) * DV + col];
    } else {
#pragma unroll
        for (int t = 0; t < DK / 16; ++t) S[t] = zero4();
    }
}

// Whole-sequence scan: one wave per (sequence, head, 16-column tile).  The
// NT waves of one (sequence, head) land on one XCD (workgroups are dealt to
// the 8 XCDs round-robin) and share the chunk operands through its L2.
template <typename T, int DK, int DV>
__global__ __launch_bounds__(64) void gdr_scan1_kernel(ScanArgs a) {
    constexpr int NT = DV / 16;
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = chain_of_rank(a, xcd + 8 * (q / NT)), tile = q % NT;
    const int H = a.n_heads;
    if (pair < 0) return;
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int64_t base = slot_base_dev(cu0, seq, a.C, a.cps);
    const size_t state_off = (size_t)pair * DK * DV;
    f32x4 S[DK / 16];
    load_state_tile<DK, DV>(start_state(a, seq, h, (size_t)DK * DV, tile == 0), tile, S);
    scan1_chunks<T, DK, DV, false>(a, seq, h, tile, len, base, nch, S, nullptr);
    if (a.final_state) {
        const int lane = threadIdx.x;
        store_state_tiles<DK / 16, DV>(a.final_state + state_off, S,
                                       4u * (uint32_t)(4 * (lane >> 4) * DV + 16 * tile + (lane & 15)));
    }
}

// Scan with output: the single-wave scan of gdr_scan1_kernel (wave 0) plus
// an output wave (wave 1) per (sequence, head, 16-column tile).  The state
// entering each chunk and U go from one wave to the other through LDS, so
// they never reach HBM, and the output product runs on another SIMD beside
// the scan's chain.
template <typename T, int DK, int DV>
__global__ __launch_bounds__(128) void gdr_scan1o_kernel(ScanArgs a) {
    constexpr int NT = DV / 16;
    __shared__ Handoff<T, DK> hs;
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = chain_of_rank(a, xcd + 8 * (q / NT)), tile = q % NT;
    const int H = a.n_heads;
    if (pair < 0) return;
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int64_t base = slot_base_dev(cu0, seq, a.C, a.cps);
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    if (wave == 0) {
        const size_t state_off = (size_t)pair * DK * DV;
        f32x4 S[DK / 16];
        load_state_tile<DK, DV>(start_state(a, seq, h, (size_t)DK * DV, tile == 0), tile, S);
        scan1_chunks<T, DK, DV, true>(a, seq, h, tile, len, base, nch, S, &hs);
        if (a.final_state) {
            const int lane = threadIdx.x & 63;
            store_state_tiles<DK / 16, DV>(a.final_state + state_off, S,
                                           4u * (uint32_t)(4 * (lane >> 4) * DV + 16 * tile + (lane & 15)));
        }
    } else {
        out_wave_chunks<T, DK, DV>(a, h, tile, cu0, len, base, nch, &hs);
    }
}

}  // namespace la

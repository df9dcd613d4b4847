// Fused chunk scan (bf16 operands): the sequential recurrence and the output
// read-out, with every chunk's keys, queries and values staged once per
// workgroup in LDS.
//
// A workgroup owns CW state columns of one (sequence, head) and runs its
// chunks in order.  Each 32 of its columns (two 16-column tiles; in the
// 32-column form each 16) belong to a pair of waves: a scan wave, which
// keeps those columns of the fp32 state in MFMA result registers for the
// whole run, and (when the unit has an output) an output wave, which reads
// the output out beside it.  Per chunk, with S_0 the state entering it
// and the gate block and X written by the preparation kernel (gdr_xprep.h):
//
//   scan wave    Y   = K S_0                      A = K rows, B = S_0
//                Z   = V - diag(exp(Gp)) Y        V in C layout
//                U   = X diag(beta) Z             A = X diag(beta) fragments, B = Z
//                S_1 = exp(G_63) S_0 + K^T diag(exp(G_63 - G)) U
//   output wave  O^T = scale ((S_0^T Q^T) diag(exp G) + U^T P^T),
//                P   = (Q K^T) exp(G_r - G_s) on s <= r, zero above
//                      (tiles dealt over the output waves, shared in LDS)
//
// Operands stay in the lanes that produce them: a C-layout result read with
// the contraction index permuted by perm_row is a B operand over its rows,
// and, transposed, an A operand over its rows.  The state's rows are held in
// a fixed permutation of dk (state_row): then the contraction order in which
// S_0 enters Y = K S_0 is plain dk order, so an A-operand fragment of K or Q
// is one 16-byte LDS read of a row, and the fragments of K^T (whose rows must
// follow the state's) are transposed LDS reads whose per-lane column
// addresses apply the same permutation.  The state handed to the output wave
// (S_0 as bf16 B-operand fragments) and U pass through LDS.
//
// Loads: a helper wave of each pair (the loader wave in the 32- and
// 64-column forms with an output, otherwise the pair's second wave) stages
// every chunk's K, Q, values and the preparation's block (X, gates) ahead:
// buffer loads into registers while earlier chunks are computed, rows past
// a chunk's end reading as zero through the buffer range, then LDS stores
// into the other of two buffers.  The scan waves issue no global loads, so
// no LDS read of theirs waits on one.
// (Loads with an LDS destination would save the registers, but every LDS
// read after them would wait for them to land.)
//
// Modes (unit = one workgroup):
//   kXScan    (sequence, head, column part): the whole sequence from its
//             starting state; output, checkpoints, final state.
//   kXReplay  (sequence, head, segment, column part): the segment's chunks
//             from the state entering it (two-level scan); output only.
//   kXMap     (sequence, head, segment, column part of [Phi | R]): the
//             segment's state map S_out = D S_in + Phi' S_in + R.  Columns of
//             Phi start from the identity and take no values, columns of R
//             start from zero; no output.
// Within a chunk every wave runs the same MFMAs in the same order whatever
// the batch, the mode or the part, so a sequence's bits do not depend on
// what it is batched with.
#pragma once
#include "gdr_scan.h"
#include "gdr_xprep.h"

#include <type_traits>

namespace la {

enum : int { kXScan = 0, kXReplay = 1, kXMap = 2 };

// Column tiles per wave (16 columns each) and wave pairs per workgroup:
// the 32-column form gives each wave one tile, the wider forms two.
constexpr int xscan_tw(int cw) { return cw == 32 ? 1 : 2; }
constexpr int xscan_npair(int cw) { return cw / (16 * xscan_tw(cw)); }
// Waves per workgroup: a scan wave and a helper per pair.  The 32- and
// 64-column forms with an output give each pair a third wave: one helper
// then reads the output out and the other (the loader) stages the inputs.
constexpr bool xscan_loaders(int cw, int mode) { return cw <= 64 && mode != kXMap; }
constexpr int xscan_threads(int cw, int mode) { return 64 * xscan_npair(cw) * (xscan_loaders(cw, mode) ? 3 : 2); }

typedef short i16x4 __attribute__((ext_vector_type(4)));

// Columns per workgroup (CW): 128 (four wave pairs of 32 columns), 64 (two)
// or 32 (two pairs of 16).  Every column's arithmetic is the same whatever
// CW, so the choice is free: narrower workgroups spread a chain over more
// CUs and shorten each chunk's step when there are few chains, 128 stages
// each chunk's K, Q and prepared block once for twice the columns.  The
// map's Phi and R parts split at a part boundary, so CW divides dk.

// dk row held at state tile-row x = 16 t + 4 g + q (lane group g, element
// q of tile t): the B-operand contraction index 8 ks + j of lane group g
// (perm_row) then stands for dk 32 ks + 8 g + j, plain order.  A lane holds
// the 8 consecutive dk rows 32 (t / 2) + 8 g .. + 7 across tiles t and t ^ 1.
__device__ __host__ inline int state_row(int x) {
    const int t = x >> 4, g = (x >> 2) & 3, q = x & 3;
    return 32 * (t >> 1) + 8 * g + 4 * (t & 1) + q;
}

template <int DK, int CW, bool OUT, int NVB> struct XLds {
    static constexpr int TW = xscan_tw(CW), NPAIR = xscan_npair(CW), PW = 16 * TW;
    static constexpr int KV = kChunk * DK / 8;   // 16-byte pieces of a chunk's K (or Q)
    struct Buf {
        uint4 k[KV];                             // K rows, pieces XOR-swizzled by row (xpiece)
        uint4 q[OUT ? KV : 1];                   // Q, same layout
        uint4 misc[kMiscVec];                    // X diag(beta) fragments, then the gate block
    };
    Buf buf[2];
    uint4 v[NVB][NPAIR][kChunk * PW / 8];        // each pair's PW value columns, row-major [64][PW]
                                                 // (double-buffered when loader waves stage them)
    uint4 pf[OUT ? 4 * 2 * 64 : 1];              // P fragments [row tile][k-step][lane]
    uint4 sbh[OUT ? NPAIR : 1][TW][DK / 32][64]; // S_0 handed to the output wave (B-operand fragments)
    uint4 ubh[OUT ? NPAIR : 1][TW][2][64];       // U handed to the output wave
};

// Physical 16-byte piece of logical piece p in row r of a K or Q tile (DK / 8
// pieces per row): the XOR swizzle spreads the rows of a fragment read over
// the LDS banks.  The plain key (r) keeps the 16 rows of a row-fragment read
// apart; the mixed key (r ^ 4 r, low bits) does too, and also spreads the
// 4 rows x 4 pieces of a K^T transposed read over 16 pieces where the plain
// key gives 4.  Measured per kernel: the mixed key speeds up the segment
// maps (no output waves) and slows the 32-column scan, so only the maps use it.
template <int DK, bool MIX> __device__ inline int xpiece(int r, int p) {
    return p ^ ((MIX ? (r ^ (r << 2)) : r) & (DK / 8 - 1));
}

// A-operand fragment of rows [16 mt, 16 mt + 16) of a K or Q tile, k-step ks
// (dk 32 ks + 8 g .. + 7): one 16-byte read.
template <int DK, bool MIX> __device__ inline bf16x8 row_frag(const uint4 *tile, int mt, int ks, int lane) {
    const int r = 16 * mt + (lane & 15), g = lane >> 4;
    return __builtin_bit_cast(bf16x8, tile[r * (DK / 8) + xpiece<DK, MIX>(r, 4 * ks + g)]);
}

// A-operand fragment of K^T for state tile t (rows state_row(16 t + i)) and
// k-step ks over the chunk rows (perm_row order: runs of 4 rows at 32 ks + 4 g
// and 32 ks + 16 + 4 g): two transposed 8-byte reads.  In each 16-lane group
// source lane s reads 4 consecutive dk columns of row base + s / 4 and lane
// 4 c + q receives column (that of source lanes c, c + 4, ...) + q of rows
// base .. base + 3, so reading the 4 columns 32 (t / 2) + 4 (t % 2) + 8 c
// gives lane 4 c + q exactly state_row(16 t + 4 c + q).
template <int DK, bool MIX> __device__ inline bf16x8 kt_frag(const uint4 *k, int t, int ks, int lane) {
    typedef short i16x8 __attribute__((ext_vector_type(8)));
    const int g = lane >> 4, s = lane & 15;
    const int piece = 4 * (t >> 1) + (s & 3), half = 8 * (t & 1);
    i16x4 h[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int r = 32 * ks + 16 * u + 4 * g + (s >> 2);
        const char *p = (const char *)k + (r * (DK / 8) + xpiece<DK, MIX>(r, piece)) * 16 + half;
        h[u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)p);
    }
    const i16x8 both = {h[0][0], h[0][1], h[0][2], h[0][3], h[1][0], h[1][1], h[1][2], h[1][3]};
    return __builtin_bit_cast(bf16x8, both);
}

// Workgroup barrier that orders LDS operations only: a workgroup release
// fence would also wait for the helper waves' global loads of the next chunk
// and the output stores in flight.
__device__ inline void xbar_lds() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
// Start state of a wave's TW column tiles (permuted rows) from a row-major
// [DK][DV] fp32 state, or zero.
template <int DK, int DV, int TW>
__device__ inline void load_state_perm(const float *src, int col0, f32x4 (&S)[TW][DK / 16]) {
    const int lane = threadIdx.x & 63, g16 = lane >> 4, c16 = lane & 15;
#pragma unroll
    for (int c = 0; c < TW; ++c)
#pragma unroll
        for (int t = 0; t < DK / 16; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                S[c][t][i] = src ? src[(size_t)state_row(16 * t + 4 * g16 + i) * DV + col0 + 16 * c + c16] : 0.f;
}

// Row-major [DK][DV] store of one column tile of the state (permuted rows);
// voff is the lane's byte offset of dk row 8 g, its column.
template <int DK, int DV>
__device__ inline void store_state_perm(float *dst, const f32x4 (&S)[DK / 16], uint32_t voff) {
    const auto r = make_rsrc(dst, DK * DV * sizeof(float));
#pragma unroll
    for (int t = 0; t < DK / 16; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_int(S[t][i]), r, (int)voff,
                                                  (32 * (t >> 1) + 4 * (t & 1) + i) * DV * (int)sizeof(float), 0);
}

template <int DK, int CW, int MODE>
using XLdsOf = XLds<DK, CW, MODE != kXMap, xscan_loaders(CW, MODE) ? 2 : 1>;

// One workgroup of the fused scan: block b of this width's blocks, whose
// units are ranked chains chain0, chain0 + 1, ... (single-level scan) or
// (sequence, head, segment) units.
template <int DK, int DV, int MODE, int CW>
__device__ __forceinline__ void xscan_block(const ScanArgs &a, XLdsOf<DK, CW, MODE> &sm, int b, int chain0) {
    using M = MT<__bf16>;
    typedef __bf16 T;
    static_assert(CW == 32 || CW == 64 || CW == 128, "column width");
    constexpr bool kOut = MODE != kXMap;
    constexpr int TW = xscan_tw(CW);                   // column tiles per wave
    constexpr int NPAIR = xscan_npair(CW);             // scan waves (and output waves with kOut)
    constexpr int PW = 16 * TW;                        // state columns per pair
    constexpr int NTH = xscan_threads(CW, MODE);
    constexpr bool kLoad3 = xscan_loaders(CW, MODE);   // loader waves of their own
    constexpr bool kMix = MODE == kXMap;               // K swizzle key (xpiece)
    constexpr int RT = DK / 16, FS = DK / 4, KS = DK / 32;
    constexpr int NCOLS = (MODE == kXMap) ? DK + DV : DV;   // column space of the unit
    constexpr int NP = NCOLS / CW;                     // parts per (sequence, head[, segment])
    static_assert(NP * CW == NCOLS && (MODE != kXMap || DK % CW == 0), "column parts");
    constexpr int NVB = kLoad3 ? 2 : 1;                // value buffers
    using Lds = XLdsOf<DK, CW, MODE>;
    constexpr int KV = Lds::KV;

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, c16 = lane & 15;
    const int role = w / NPAIR;                        // 0 scan, 1 helper, 2 loader (kLoad3)
    const bool scan_wave = role == 0;
    const int pr = w % NPAIR;                          // the wave's pair
    const int H = a.n_heads;

    // ---- unit: (sequence, head[, segment], part); the parts of one chain
    // (or segment) share an XCD and its L2
    int pair, sg = 0;
    const int xcd = b & 7, qb = b >> 3;
    const int part = qb % NP, chain = chain0 + xcd + 8 * (qb / NP);
    if constexpr (MODE == kXScan) {
        pair = chain_of_rank(a, chain);
        if (pair < 0) return;
    } else {
        if (chain >= a.n_seqs * H * a.max_seg) return;
        pair = chain / a.max_seg;
        sg = chain % a.max_seg;
    }
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int64_t base = slot_base_dev(cu0, seq, a.C, a.cps);
    int c0 = 0, c1 = nch;
    int64_t seg_slot = 0;
    if constexpr (MODE != kXScan) {
        c0 = sg * a.seg_m;
        if (c0 >= nch) return;
        c1 = min(c0 + a.seg_m, nch);
        seg_slot = slot_base_dev(cu0, seq, (int64_t)a.C * a.seg_m, a.cps) + sg;
    }
    const int cb = part * CW;                          // first column of the part
    const bool phi = MODE == kXMap && cb < DK;         // a part of Phi (identity start, no values)
    const int vcol0 = (MODE == kXMap) ? cb - DK : cb;  // first value (state) column of the part
    const int pcol = vcol0 + PW * pr;                  // first state column of the wave's pair

    // ---- staging of chunk jj's inputs by the helper waves (the loader
    // waves, or without them the pairs' second waves): global loads into
    // registers (rows past the chunk's end read as zero through the buffer
    // range), then 16-byte LDS stores.  Helper wave p stages its share of K,
    // Q, the preparation's block and the workgroup's CW value columns (those
    // taken row by row across all pairs, so that each load instruction reads
    // whole CW-column row pieces rather than one pair's PW columns).  The scan
    // waves issue no global loads, so nothing they read from LDS waits on a
    // load in flight.
    constexpr int KPW = KV / 64 / NPAIR;                 // 16-byte pieces of K per helper lane
    constexpr int MPW = (kMiscVec + 64 * NPAIR - 1) / (64 * NPAIR);
    constexpr int VPR = PW / 8;                          // 16-byte pieces of a value row of a pair
    constexpr int VPC = CW / 8;                          // 16-byte pieces of a value row of the workgroup
    constexpr int VPW = kChunk * VPC / 64 / NPAIR;       // pieces of the values per helper lane
    static_assert(VPW * 64 * NPAIR == kChunk * VPC, "value staging tiling");
    constexpr int VROWS = 64 / VPC, VLP = 64 / NPAIR;    // rows per value load; lanes per pair
    auto vrow = [&](int it) { return (pr * VPW + it) * VROWS + (lane % VLP) / VPR; };
    auto vpiece = [&]() { return (lane / VLP) * VPR + lane % VPR; };
    static_assert(KPW * 64 * NPAIR == KV, "K staging tiling");
    struct Stage {
        uint4 k[KPW], q[kOut ? KPW : 1], m[MPW], v[VPW];
    };
    const T *qin = (const T *)a.q, *kin = (const T *)a.k, *vin = (const T *)a.v;
    const bool has_v = !phi;
    // A chunk past the run's last has empty ranges: its loads read zero and
    // touch no memory, so a loader can issue them unconditionally.
    auto stage_load = [&](Stage &st, int jj) {
        const bool live = jj < c1;
        int lo = 0, hi = 0;
        if (live) chunk_range32(jj, len, a.C, a.cps, &lo, &hi);
        const int n = hi - lo;
        const int64_t row0 = ((int64_t)cu0 + lo) * H + h;
        const uint32_t rows_k = live ? head_rows_bytes<T>(n, H, DK) : 0u;
        const auto rk = make_rsrc(kin + row0 * DK, rows_k);
        const auto rq = make_rsrc(qin + row0 * DK, rows_k);
#pragma unroll
        for (int it = 0; it < KPW; ++it) {
            const int e = (pr * KPW + it) * 64 + lane, r = e / (DK / 8), p = e % (DK / 8);
            const uint32_t voff = (uint32_t)(r * H * DK * 2 + 16 * p);
            st.k[it] = buf_load16(rk, voff, 0u);
            if constexpr (kOut) st.q[it] = buf_load16(rq, voff, 0u);
        }
        const auto rm = make_rsrc(a.ws.misc + ((base + jj) * H + h) * kMiscVec, live ? kMiscVec * 16 : 0u);
#pragma unroll
        for (int it = 0; it < MPW; ++it)
            st.m[it] = buf_load16(rm, (uint32_t)(((pr * MPW + it) * 64 + lane) * 16), 0u);
        const uint32_t vbytes =
            (has_v && live) ? (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)((n - 1) * H * DV + CW) * 2)) : 0u;
        const auto rv = make_rsrc(vin + row0 * DV + vcol0, vbytes);
#pragma unroll
        for (int it = 0; it < VPW; ++it) {
            const int r = vrow(it), p = vpiece();
            st.v[it] = buf_load16(rv, (uint32_t)(r * H * DV * 2 + 16 * p), 0u);
        }
    };
    auto stage_store_shared = [&](const Stage &st, int bi) {
        typename Lds::Buf &B = sm.buf[bi];
#pragma unroll
        for (int it = 0; it < KPW; ++it) {
            const int e = (pr * KPW + it) * 64 + lane, r = e / (DK / 8), p = e % (DK / 8);
            B.k[r * (DK / 8) + xpiece<DK, kMix>(r, p)] = st.k[it];
            if constexpr (kOut) B.q[r * (DK / 8) + xpiece<DK, kMix>(r, p)] = st.q[it];
        }
#pragma unroll
        for (int it = 0; it < MPW; ++it) {
            const int e = (pr * MPW + it) * 64 + lane;
            if (e < kMiscVec) B.misc[e] = st.m[it];
        }
    };
    // Each of the helper's value loads covers VROWS whole rows of the
    // workgroup's CW columns: lane l takes pair l / (64 / NPAIR), so that the
    // lanes of one pair store a contiguous run of that pair's row-major
    // [64][PW] block.
    auto stage_store_values = [&](const Stage &st, int bi) {
        uint4 *vb = &sm.v[bi % NVB][0][0];
#pragma unroll
        for (int it = 0; it < VPW; ++it) {
            const int r = vrow(it), p = vpiece();
            vb[(p / VPR) * (kChunk * VPR) + r * VPR + p % VPR] = st.v[it];
        }
    };

    // P fragments above the diagonal that no P tile writes stay zero
    if constexpr (kOut) {
        for (int e = tid; e < 4 * 2 * 64; e += NTH) sm.pf[e] = make_uint4(0, 0, 0, 0);
    }

    if (scan_wave) {
        // ================================ scan wave ================================
        // the chain: ahead of the helper that shares this wave's SIMD
        __builtin_amdgcn_s_setprio(2);
        f32x4 S[TW][RT];
        if constexpr (MODE == kXMap) {
#pragma unroll
            for (int c = 0; c < TW; ++c)
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        S[c][t][i] = (phi && state_row(16 * t + 4 * g16 + i) == cb + PW * pr + 16 * c + c16) ? 1.f : 0.f;
        } else if (MODE == kXReplay && sg > 0) {
            const float *src = a.seg.state + (seg_slot * H + h) * DK * DV;
#pragma unroll
            for (int c = 0; c < TW; ++c) load_state_c<RT>(src, pcol / 16 + c, S[c]);
        } else {
            load_state_perm<DK, DV>(start_state(a, seq, h, (size_t)DK * DV, part == 0 && pr == 0), pcol, S);
        }
        float dprod = 1.f;   // product of the chunk decays (the map's D)
        CkptDst ck;
        if constexpr (MODE == kXScan) {
            ck.init(a, seq, h, len, (size_t)DK * DV, part == 0 && pr == 0);
            ck.load_window(0);
        }
        uint32_t soff[TW];
#pragma unroll
        for (int c = 0; c < TW; ++c) soff[c] = 4u * (uint32_t)(8 * g16 * DV + pcol + 16 * c + c16);

        // S_0 as bf16 B operand (k-step ks: dk 32 ks + 8 g .. + 7)
        T sb[TW][FS];
        auto make_sb = [&]() {
#pragma unroll
            for (int c = 0; c < TW; ++c)
#pragma unroll
                for (int f = 0; f < FS; ++f) sb[c][f] = (T)S[c][f >> 2][f & 3];
            if constexpr (kOut) {
#pragma unroll
                for (int c = 0; c < TW; ++c)
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) sm.sbh[pr][c][ks][lane] = *(const uint4 *)&sb[c][8 * ks];
            }
        };
        make_sb();
        xbar_lds();

        for (int jj = c0; jj < c1; ++jj) {
            const int bi = (jj - c0) & 1;
            const typename Lds::Buf &B = sm.buf[bi];
            int lo, hi;
            chunk_range32(jj, len, a.C, a.cps, &lo, &hi);

            // Each phase issues its LDS reads ahead of the MFMAs that use them
            // (sched_barrier keeps the order): one wave per SIMD pair half
            // cannot hide LDS latency otherwise.
            // ---- Y = K S_0: row tiles 0-1's K fragments in flight, then 2-3's
            // behind the first half of the MFMAs
            const float *gate = (const float *)&B.misc[kXFrags * 64];
            bf16x8 kf[4][KS];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) kf[mt][ks] = row_frag<DK, kMix>(B.k, mt, ks, lane);
            const float eL = __builtin_amdgcn_exp2f(gate[kChunk - 1] * kLog2e);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mt = 2; mt < 4; ++mt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) kf[mt][ks] = row_frag<DK, kMix>(B.k, mt, ks, lane);
            f32x4 Y[TW][4];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int c = 0; c < TW; ++c) {
                    Y[c][mt] = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) Y[c][mt] = M::mma(kf[mt][ks], M::pack(&sb[c][8 * ks]), Y[c][mt]);
                }
            __builtin_amdgcn_sched_barrier(0);
            // the reads of Z and U (values, gates, X) behind the second half of Y
            float4 d4[4];   // exp(Gp) of the lane's rows
            i16x4 vr[TW][4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                d4[mt] = *(const float4 *)&gate[kChunk + 16 * mt + 4 * g16];
#pragma unroll
                for (int c = 0; c < TW; ++c)
                    vr[c][mt] = RowTile<T>::tr4((const T *)&sm.v[bi % NVB][pr][0], PW, 16 * mt + 4 * g16 + ((lane & 15) >> 2), 16 * c, lane);
            }
            bf16x8 xf[kXFrags];
#pragma unroll
            for (int e = 0; e < kXFrags; ++e) xf[e] = __builtin_bit_cast(bf16x8, B.misc[e * 64 + lane]);
            // exp(G_63) S_0, the state update's starting accumulator, while the
            // MFMAs of Y run (Y reads S_0 from its bf16 copy)
#pragma unroll
            for (int c = 0; c < TW; ++c)
#pragma unroll
                for (int t = 0; t < RT; ++t) S[c][t] = S[c][t] * eL;
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mt = 2; mt < 4; ++mt)
#pragma unroll
                for (int c = 0; c < TW; ++c) {
                    Y[c][mt] = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) Y[c][mt] = M::mma(kf[mt][ks], M::pack(&sb[c][8 * ks]), Y[c][mt]);
                }
            __builtin_amdgcn_sched_barrier(0);
            // the K^T fragments of the state update's first half, in flight behind Z
            bf16x8 kt[RT][2];
#pragma unroll
            for (int t = 0; t < RT / 2; ++t)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) kt[t][ks] = kt_frag<DK, kMix>(B.k, t, ks, lane);
            __builtin_amdgcn_sched_barrier(0);
            // ---- Z = V - diag(exp(Gp)) Y; U = X diag(beta) Z
            T zb[TW][16];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const float dv[4] = {d4[mt].x, d4[mt].y, d4[mt].z, d4[mt].w};
#pragma unroll
                for (int c = 0; c < TW; ++c)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        zb[c][4 * mt + i] =
                            (T)__builtin_fmaf(-dv[i], Y[c][mt][i], (float)__builtin_bit_cast(T, (short)vr[c][mt][i]));
            }
            __builtin_amdgcn_sched_barrier(0);
            // the second half's K^T fragments, in flight behind U
#pragma unroll
            for (int t = RT / 2; t < RT; ++t)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) kt[t][ks] = kt_frag<DK, kMix>(B.k, t, ks, lane);
            __builtin_amdgcn_sched_barrier(0);
            f32x4 U[TW][4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int c = 0; c < TW; ++c) {
                    U[c][mt] = zero4();
#pragma unroll
                    for (int ks = 0; ks <= (mt >> 1); ++ks)
                        U[c][mt] = M::mma(xf[xfrag_slot(mt, ks)], M::pack(&zb[c][8 * ks]), U[c][mt]);
                }
            // ---- U to the output wave (unscaled), and diag(exp(G_63 - G)) U
            T ub2[TW][16];
            {
                float4 e4[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) e4[mt] = *(const float4 *)&gate[3 * kChunk + 16 * mt + 4 * g16];
                T ub[TW][16];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const float ev[4] = {e4[mt].x, e4[mt].y, e4[mt].z, e4[mt].w};
#pragma unroll
                    for (int c = 0; c < TW; ++c)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            ub[c][4 * mt + i] = (T)U[c][mt][i];
                            ub2[c][4 * mt + i] = (T)(U[c][mt][i] * ev[i]);
                        }
                }
                if constexpr (kOut) {
#pragma unroll
                    for (int c = 0; c < TW; ++c)
#pragma unroll
                        for (int ks = 0; ks < 2; ++ks) sm.ubh[pr][c][ks][lane] = *(const uint4 *)&ub[c][8 * ks];
                }
                xbar_lds();   // B_jj: U handed off (the output waves' P tiles are written); the
                              // values of chunk jj are read, so the helpers may replace them
            }
            // ---- S = exp(G_63) S + K^T diag(exp(G_63 - G)) U
            dprod *= eL;
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int c = 0; c < TW; ++c) {
                    f32x4 acc = S[c][t];
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) acc = M::mma(kt[t][ks], M::pack(&ub2[c][8 * ks]), acc);
                    S[c][t] = acc;
                }
            if constexpr (MODE == kXScan) {
                // checkpoint when the chunk ends on a multiple of C (positions are
                // local and start on a multiple of C)
                if (hi % a.C == 0) {
                    if (float *d = ck.next(ck.window_id(hi / a.C - 1))) {
#pragma unroll
                        for (int c = 0; c < TW; ++c) store_state_perm<DK, DV>(d, S[c], soff[c]);
                    }
                }
            }
            make_sb();
            xbar_lds();   // C_jj: chunk jj + 1's inputs and the state handoff are in LDS
        }

        // ---- epilogue
        if constexpr (MODE == kXScan) {
            if (a.final_state) {
#pragma unroll
                for (int c = 0; c < TW; ++c)
                    store_state_perm<DK, DV>(a.final_state + (size_t)pair * DK * DV, S[c], soff[c]);
            }
        }
        if constexpr (MODE == kXMap) {
            const int64_t ssh = seg_slot * H + h;
#pragma unroll
            for (int c = 0; c < TW; ++c) {
                const int col = cb + PW * pr + 16 * c + c16;
                if (phi) {
                    // Phi' = Phi - D I in the io type, stored as the combine's A-operand
                    // fragments: [tile t][k-step ks][lane 16 g + c][8], row
                    // state_row(16 t + c), columns 32 ks + 8 g .. + 7, so that each of
                    // the combine's fragment loads is 1 KB contiguous.  This lane holds
                    // rows state_row(16 t + 4 g16 + e) of column col.
                    T *dst = (T *)a.seg.phi + ssh * DK * DK;
                    const int fks = col >> 5, fg = (col >> 3) & 3, fj = col & 7;
#pragma unroll
                    for (int t = 0; t < RT; ++t)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int r = state_row(16 * t + 4 * g16 + e);
                            dst[((size_t)(t * KS + fks) * 64 + 16 * fg + 4 * g16 + e) * 8 + fj] =
                                (T)(S[c][t][e] - (r == col ? dprod : 0.f));
                        }
                } else {
                    float4 *dst = (float4 *)(a.seg.r + ssh * DK * DV);
                    const int tile = (col - DK) / 16;
#pragma unroll
                    for (int t = 0; t < RT; ++t)
                        dst[(tile * RT + t) * 64 + lane] = make_float4(S[c][t][0], S[c][t][1], S[c][t][2], S[c][t][3]);
                }
            }
            if (part == 0 && pr == 0 && lane == 0) a.seg.d[ssh] = dprod;
        }
    } else if (role == 2) {
        // ================================ loader wave ================================
        // (kLoad3) Two register sets, by chunk parity P: during chunk jj the
        // loader issues the global loads of chunk jj + 2 into set P (whose
        // chunk jj is already in LDS) before B_jj, and after B_jj, beside the
        // state update, stores chunk jj + 1 (set P ^ 1, loaded during chunk
        // jj - 1) into the other LDS buffers, last read in chunk jj - 1.
        if constexpr (kLoad3) {
            Stage st[2];
            stage_load(st[0], c0);
            stage_store_shared(st[0], 0);
            stage_store_values(st[0], 0);
            stage_load(st[1], c0 + 1);
            xbar_lds();
            auto chunk = [&](auto parity, int jj) __attribute__((always_inline)) {
                constexpr int P = decltype(parity)::value;
                stage_load(st[P], jj + 2);   // unconditional: st[P] is dead until then
                xbar_lds();   // B_jj
                if (jj + 1 < c1) {
                    stage_store_shared(st[P ^ 1], P ^ 1);
                    stage_store_values(st[P ^ 1], P ^ 1);
                }
                xbar_lds();   // C_jj
            };
            for (int jj = c0; jj < c1; jj += 2) {
                chunk(std::integral_constant<int, 0>{}, jj);
                if (jj + 1 < c1) chunk(std::integral_constant<int, 1>{}, jj + 1);
            }
        }
    } else {
        // ============================ helper (output) wave ============================
        // Reads the output out and, without loader waves, stages every
        // chunk's inputs one chunk ahead.
        [[maybe_unused]] Stage st;
        if constexpr (!kLoad3) {
            stage_load(st, c0);
            stage_store_shared(st, 0);
            stage_store_values(st, 0);
        }
        xbar_lds();
        [[maybe_unused]] const float scale = a.scale;
        for (int jj = c0; jj < c1; ++jj) {
            const int bi = (jj - c0) & 1;
            const typename Lds::Buf &B = sm.buf[bi];
            int lo, hi;
            chunk_range32(jj, len, a.C, a.cps, &lo, &hi);
            [[maybe_unused]] const int n = hi - lo;
            [[maybe_unused]] const float *gate = (const float *)&B.misc[kXFrags * 64];
            if constexpr (!kLoad3) {
                if (jj + 1 < c1) stage_load(st, jj + 1);
            }
            [[maybe_unused]] f32x4 O[TW][4];   // S_0^T Q^T, finished after B_jj
            if constexpr (kOut) {
                // S_0 handed over at the end of the previous chunk, the Q fragments
                // and the K fragments of this wave's P tiles, all in flight first.
                // P tiles (mt, nt), nt <= mt: tile index mt (mt + 1) / 2 + nt,
                // dealt to the output waves round-robin.
                bf16x8 sb[TW][KS], qf[4][KS];
#pragma unroll
                for (int c = 0; c < TW; ++c)
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) sb[c][ks] = __builtin_bit_cast(bf16x8, sm.sbh[pr][c][ks][lane]);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) qf[mt][ks] = row_frag<DK, kMix>(B.q, mt, ks, lane);
                // K fragments of this wave's P tiles: column block nt = pr (and
                // nt = 0 for the tile (3, 0) the last wave takes over)
                bf16x8 pk[KS], pk0[KS];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) pk[ks] = row_frag<DK, kMix>(B.k, pr, ks, lane);
                if (pr == NPAIR - 1 && NPAIR > 1) {
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) pk0[ks] = row_frag<DK, kMix>(B.k, 0, ks, lane);
                }
                __builtin_amdgcn_sched_barrier(0);
                // ---- S_0^T Q^T
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int c = 0; c < TW; ++c) {
                        O[c][mt] = zero4();
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) O[c][mt] = M::mma(sb[c][ks], qf[mt][ks], O[c][mt]);
                    }
                // ---- P tiles (mt, nt), nt <= mt, lane (g, c) holding
                // P[r = 16 mt + c][s = 16 nt + 4 g + i]: wave p takes the tiles of
                // column block p (with NPAIR = 4 the tile (3, 0) moves from wave 0
                // to wave 3, which balances them 3, 3, 2, 2); with two waves, five
                // tiles each.
                auto p_tile = [&](int mt, int nt, const bf16x8 (&kk)[KS], const bf16x8 (&qq)[KS]) {
                    f32x4 p = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) p = M::mma(kk[ks], qq[ks], p);
                    const float gr = gate[16 * mt + c16] * kLog2e;
                    const float4 gs = *(const float4 *)&gate[16 * nt + 4 * g16];
                    const float gsv[4] = {gs.x, gs.y, gs.z, gs.w};
                    T pv[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int s_ = 16 * nt + 4 * g16 + e, r = 16 * mt + c16;
                        pv[e] = (T)(s_ <= r ? p[e] * __builtin_amdgcn_exp2f(gr - gsv[e] * kLog2e) : 0.f);
                    }
                    *(uint2 *)((char *)&sm.pf[(2 * mt + (nt >> 1)) * 64 + lane] + 8 * (nt & 1)) = *(const uint2 *)pv;
                };
                if constexpr (NPAIR == 4) {
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) {
                        if (mt >= pr && !(pr == 0 && mt == 3)) p_tile(mt, pr, pk, qf[mt]);   // wave-uniform
                    }
                    if (pr == 3) p_tile(3, 0, pk0, qf[3]);
                } else {
                    // two waves, five tiles each: wave 0 column block 0 and the
                    // tile (1, 1), wave 1 the rest of column blocks 1..3
                    if (pr == 0) {
#pragma unroll
                        for (int mt = 0; mt < 4; ++mt) p_tile(mt, 0, pk, qf[mt]);
                        bf16x8 kk[KS];
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) kk[ks] = row_frag<DK, kMix>(B.k, 1, ks, lane);
                        p_tile(1, 1, kk, qf[1]);
                    } else {
#pragma unroll
                        for (int mt = 2; mt < 4; ++mt) p_tile(mt, 1, pk, qf[mt]);
#pragma unroll
                        for (int nt = 2; nt < 4; ++nt) {
                            bf16x8 kk[KS];
#pragma unroll
                            for (int ks = 0; ks < KS; ++ks) kk[ks] = row_frag<DK, kMix>(B.k, nt, ks, lane);
#pragma unroll
                            for (int mt = nt; mt < 4; ++mt) p_tile(mt, nt, kk, qf[mt]);
                        }
                    }
                }
            }
            xbar_lds();   // B_jj
            if constexpr (kOut) {
                // ---- O^T = scale ((S_0^T Q^T) diag(exp G) + U^T P^T), 4 columns per lane
                bf16x8 ubf[TW][2], pfr[kXFrags];
#pragma unroll
                for (int c = 0; c < TW; ++c)
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) ubf[c][ks] = __builtin_bit_cast(bf16x8, sm.ubh[pr][c][ks][lane]);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int ks = 0; ks <= (mt >> 1); ++ks)
                        pfr[xfrag_slot(mt, ks)] = __builtin_bit_cast(bf16x8, sm.pf[(2 * mt + ks) * 64 + lane]);
                float eg[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) eg[mt] = __builtin_amdgcn_exp2f(gate[16 * mt + c16] * kLog2e);
                __builtin_amdgcn_sched_barrier(0);
                T *obase = (T *)a.o + (((int64_t)cu0 + lo) * H + h) * DV;
                [[maybe_unused]] const auto ro = make_rsrc(obase, head_rows_bytes<T>(n, H, DV));
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    uint2 out[TW];   // 4 bf16 columns of row 16 mt + c16 per tile
#pragma unroll
                    for (int c = 0; c < TW; ++c) {
                        f32x4 acc = O[c][mt] * eg[mt];
#pragma unroll
                        for (int ks = 0; ks <= (mt >> 1); ++ks) acc = M::mma(ubf[c][ks], pfr[xfrag_slot(mt, ks)], acc);
                        T o4[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) o4[e] = (T)(acc[e] * scale);
                        out[c] = *(const uint2 *)o4;
                    }
                    if constexpr (CW == 128) {
                        // Lane groups g and g ^ 1 trade halves (ds_swizzle, lane ^ 16
                        // within 32) so that even groups hold 8 consecutive columns of
                        // tile 0 and odd groups 8 of tile 1: one 16-byte store per lane,
                        // 64 contiguous bytes per row instead of two 32-byte pieces.
                        // Without loader waves the output wave's stores queue ahead of
                        // its next staging loads, so halving them shortens its chunk
                        // (the 64-column form, whose loaders issue those loads, is
                        // measured slower with it).
                        const bool odd = g16 & 1;
                        const uint2 send = odd ? out[0] : out[1];
                        const uint2 recv = make_uint2((uint32_t)__builtin_amdgcn_ds_swizzle((int)send.x, 0x401F),
                                                      (uint32_t)__builtin_amdgcn_ds_swizzle((int)send.y, 0x401F));
                        const uint4 v = odd ? make_uint4(recv.x, recv.y, out[1].x, out[1].y)
                                            : make_uint4(out[0].x, out[0].y, recv.x, recv.y);
                        const int row = 16 * mt + c16;
                        if (row < n)
                            *(uint4 *)(obase + (int64_t)row * H * DV + pcol + 16 * (g16 & 1) + 8 * (g16 >> 1)) = v;
                    } else {
#pragma unroll
                        for (int c = 0; c < TW; ++c) {
                            const uint32_t voff = ((uint32_t)(16 * mt + c16) * (uint32_t)(H * DV) +
                                                   (uint32_t)(pcol + 16 * c + 4 * g16)) * (uint32_t)sizeof(T);
                            buf_store8(out[c], ro, voff, 0u);
                        }
                    }
                }
            }
            // chunk jj + 1's inputs: the other buffers were last read in chunk
            // jj - 1
            if constexpr (!kLoad3) {
                if (jj + 1 < c1) {
                    stage_store_shared(st, bi ^ 1);
                    stage_store_values(st, bi ^ 1);
                }
            }
            xbar_lds();   // C_jj
        }
    }
}

template <int DK, int DV, int MODE, int CW>
__global__ __launch_bounds__((xscan_threads(CW, MODE))) void gdr_xscan_kernel(ScanArgs a) {
    __shared__ XLdsOf<DK, CW, MODE> sm;
    xscan_block<DK, DV, MODE, CW>(a, sm, blockIdx.x, 0);
}

// Single-level scan at two widths in one launch: the a.n_narrow longest
// ranked chains (a multiple of 8) in 32-column workgroups (blocks first),
// the others in 64-column workgroups.  Both forms have 384 threads and
// share one LDS allocation.
template <int DK, int DV>
__global__ __launch_bounds__(384) void gdr_xscan_mixed_kernel(ScanArgs a) {
    using L32 = XLdsOf<DK, 32, kXScan>;
    using L64 = XLdsOf<DK, 64, kXScan>;
    static_assert(xscan_threads(32, kXScan) == 384 && xscan_threads(64, kXScan) == 384, "one block size");
    __shared__ __attribute__((aligned(16))) unsigned char raw[sizeof(L32) > sizeof(L64) ? sizeof(L32) : sizeof(L64)];
    const int nb32 = 4 * a.n_narrow;   // 8 * (DV / 32) blocks per 8 chains
    if ((int)blockIdx.x < nb32)
        xscan_block<DK, DV, kXScan, 32>(a, *reinterpret_cast<L32 *>(raw), blockIdx.x, 0);
    else
        xscan_block<DK, DV, kXScan, 64>(a, *reinterpret_cast<L64 *>(raw), blockIdx.x - nb32, a.n_narrow);
}

// Two-level scan, second level: per (sequence, head, 16-column tile), the
// segment states in order, S <- D S + Phi' S + R (the large D I part stays
// in fp32; only Phi' S goes through the bf16 MFMA).  The state's rows are
// held in the fused scan's permutation (state_row), as are R and the
// segment-entering states it exchanges with the map and the replay; Phi' is
// in the A-operand fragment order the map writes.  Writes the checkpoints (segment ends on a multiple of
// C), the state entering every later segment, and the final state.
//
// One wave per 32 state rows (row tiles 2w, 2w + 1): those two tiles of S,
// in bf16, are exactly k-step w of the B operand of Phi' S, so each wave
// hands its fragment to the others through LDS (double-buffered by segment
// parity, one barrier per segment) and computes its own rows of the next
// state; a segment step is then 2 KS MFMAs per wave instead of RT KS on one.
template <int DK, int DV>
__global__ __launch_bounds__(64 * (DK / 32)) void gdr_xcombine_kernel(ScanArgs a) {
    using M = MT<__bf16>;
    typedef __bf16 T;
    constexpr int RT = DK / 16, NT = DV / 16, KS = DK / 32;
    constexpr int kMfmas = 2 * KS, kLoads = 1 + 2 + 2 * KS;
    __shared__ uint4 sbs[2][KS][64];   // the state's B-operand fragments [segment parity][k-step][lane]
    const int lane = threadIdx.x & 63, g16 = lane >> 4, c16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));   // row tiles 2w, 2w + 1
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = chain_of_rank(a, xcd + 8 * (q / NT)), tile = q % NT;
    const int H = a.n_heads;
    if (pair < 0) return;
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int nseg = (nch + a.seg_m - 1) / a.seg_m;
    const int64_t sbase = slot_base_dev(cu0, seq, (int64_t)a.C * a.seg_m, a.cps);
    const int col = 16 * tile + c16;
    f32x4 S[2];
    {
        const float *src = start_state(a, seq, h, (size_t)DK * DV, tile == 0 && w == 0);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                S[u][i] = src ? src[(size_t)state_row(16 * (2 * w + u) + 4 * g16 + i) * DV + col] : 0.f;
    }
    CkptDst ck;
    ck.init(a, seq, h, len, (size_t)DK * DV, tile == 0 && w == 0);
    // the lane's byte offset of its first row (32 w + 8 g) and its column
    const uint32_t soff = 4u * (uint32_t)((32 * w + 8 * g16) * DV + col);
    // rows of this wave's tiles, row-major [DK][DV]: 32 w + 8 g + 4 u + i
    auto store_rows = [&](float *dst) {
        const auto r = make_rsrc(dst, DK * DV * sizeof(float));
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_int(S[u][i]), r, (int)soff,
                                                      (4 * u + i) * DV * (int)sizeof(float), 0);
    };
    __builtin_amdgcn_s_waitcnt(0);

    struct Ops {
        float d;
        int ckid;             // page id of the checkpoint this segment would end (paged)
        f32x4 r[2];
        uint4 ph[2][KS];
    };
    auto load = [&](Ops &o, int sg) {
        const int64_t ssh = (sbase + sg) * H + h;
        o.ckid = ck.load_id(max((sg + 1) * a.seg_m / a.cps - 1, 0));
        o.d = buf_load4f(make_rsrc(a.seg.d + ssh, sizeof(float)), 0u, 0u);
        const auto rr = make_rsrc(a.seg.r + ssh * DK * DV, DK * DV * sizeof(float));
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const uint4 x = buf_load16(rr, 16u * lane, 1024u * (tile * RT + 2 * w + u));
            o.r[u] = f32x4{__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z), __uint_as_float(x.w)};
        }
        // A operand of Phi' for state tile t (row state_row(16 t + c), dk 32 ks + 8 g .. + 7),
        // stored by the map in fragment order: one contiguous 1 KB load each
        const auto rp = make_rsrc((const T *)a.seg.phi + ssh * DK * DK, DK * DK * sizeof(T));
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                o.ph[u][ks] = buf_load16(rp, 16u * lane, (uint32_t)(((2 * w + u) * KS + ks) * 1024));
    };
    auto step = [&](const Ops &o, int sg) {
        // this wave's k-step of S as bf16, to every wave
        T sb[8];
#pragma unroll
        for (int f = 0; f < 8; ++f) sb[f] = (T)S[f >> 2][f & 3];
        sbs[sg & 1][w][lane] = *(const uint4 *)sb;
        xbar_lds();
        bf16x8 bf[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) bf[ks] = __builtin_bit_cast(bf16x8, sbs[sg & 1][ks][lane]);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            f32x4 acc = S[u] * o.d + o.r[u];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) acc = M::mma(__builtin_bit_cast(bf16x8, o.ph[u][ks]), bf[ks], acc);
            S[u] = acc;
        }
#pragma unroll
        for (int i = 0; i < kMfmas; ++i) {
            if (i < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        if (kLoads > kMfmas) __builtin_amdgcn_sched_group_barrier(0x020, kLoads - kMfmas, 0);
        int lo, hi;
        chunk_range32(min((sg + 1) * a.seg_m, nch) - 1, len, a.C, a.cps, &lo, &hi);
        if (sg + 1 < nseg) {
            float4 *st = (float4 *)(a.seg.state + ((sbase + sg + 1) * H + h) * DK * DV);
#pragma unroll
            for (int u = 0; u < 2; ++u)
                st[(tile * RT + 2 * w + u) * 64 + lane] = make_float4(S[u][0], S[u][1], S[u][2], S[u][3]);
        }
        if (hi % a.C == 0) {   // checkpoints come in order, one per C-aligned segment end
            if (float *d = ck.next(o.ckid)) store_rows(d);
        }
    };
    scan_ring<1>(nseg, load, step, (Ops *)nullptr);
    if (a.final_state) store_rows(a.final_state + (size_t)pair * DK * DV);
}

}  // namespace la

// Workgroup forms of the chunk scan for the two-level scan's parallel
// levels, for throughput: the chunk operands (-W and K~^T, 32 KB per chunk
// at dk = 128) are read from HBM/L2 once per workgroup and shared through
// LDS, instead of once per 16-column wave.
//
// A workgroup owns one unit of state columns:
//   kGroupTrans   (sequence, head, segment), DK + DV columns of [Phi | R]
//                 started from [I | 0]: the segment's state map;
//   kGroupReplay  (sequence, head, segment), DV columns from the segment's
//                 entering state: the state entering each chunk and U.
// Its 4 waves own TPW tiles each (tile i of wave w is column tile
// i * 4 + w; with that striding a wave's Phi tiles are its first DK/64).
// Per chunk j, every wave
//   1. writes its quarter of chunk j+1's operands (loaded during chunk j-1)
//      into the LDS buffer (j+1) & 1 and issues the global loads of its
//      quarter of chunk j+2;
//   2. computes chunk j from buffer j & 1: each operand fragment is read from
//      LDS once and used for all TPW tiles;
//   3. meets the others at one barrier.
#pragma once
#include "gdr_scan.h"

namespace la {

enum : int { kGroupTrans = 1, kGroupReplay = 2 };
constexpr int kGroupWaves = 4;

template <typename T, int DK> struct GroupOps {
    static constexpr int VEC = Vec<T>::N;
    static constexpr int VS = DK / 4 / VEC;               // -W vectors per row tile
    static constexpr int VU = kChunk / 4 / VEC;           // K~^T vectors per row tile
    static constexpr int NW = 4 * VS;                     // -W vectors per chunk
    static constexpr int NV = NW + (DK / 16) * VU;        // all vectors (1 KB each)
    static constexpr int PER_WAVE = NV / kGroupWaves;
    static_assert(NW == (DK / 16) * VU && PER_WAVE * kGroupWaves == NV, "operand split");
};

template <typename T, int DK, int DV, int MODE>
__global__ __launch_bounds__(64 * kGroupWaves) void gdr_group_kernel(ScanArgs a) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    using G = GroupOps<T, DK>;
    constexpr int KW = M::KW, VEC = G::VEC, VS = G::VS, VU = G::VU, NV = G::NV, PW = G::PER_WAVE;
    constexpr int RT = DK / 16, FS = DK / 4, FU = kChunk / 4;
    constexpr int NTU = (MODE == kGroupTrans) ? (DK + DV) / 16 : DV / 16;   // tiles per unit
    constexpr int TPW = NTU / kGroupWaves;
    constexpr int NPHI = (MODE == kGroupTrans) ? DK / 64 : 0;               // Phi tiles per wave
    constexpr bool kHandOff = MODE != kGroupTrans;
    static_assert(TPW * kGroupWaves == NTU, "tiles per wave");
    constexpr int kMfmas = TPW * (4 * VS + RT * VU) * (VEC / KW);     // per chunk
    constexpr int kLoads = PW + 1 + 4 * (TPW - NPHI);                  // global loads per chunk

    __shared__ uint4 ops_lds[2][NV][64];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, c16 = lane & 15;
    const int H = a.n_heads;
    // unit -> (sequence, head[, segment]); units of consecutive ids go to
    // consecutive XCDs
    int seq, h, seg = 0, len, nch, c0, c1;
    int64_t base, seg_slot = 0;
    {
        const int unit = blockIdx.x;
        const int pair = unit / a.max_seg;
        seg = unit % a.max_seg;
        if (pair >= a.n_seqs * H) return;
        seq = pair / H;
        h = pair % H;
        const int cu0 = a.cu[seq];
        len = a.cu[seq + 1] - cu0;
        nch = n_chunks32(len, a.C, a.cps);
        base = slot_base_dev(cu0, seq, a.C, a.cps);
        c0 = seg * a.seg_m;
        if (c0 >= nch) return;
        c1 = min(c0 + a.seg_m, nch);
        seg_slot = slot_base_dev(cu0, seq, (int64_t)a.C * a.seg_m, a.cps) + seg;
    }
    const int n = c1 - c0;

    // ---- initial state of every tile
    f32x4 S[TPW][RT];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tile = i * kGroupWaves + w;
        if (MODE == kGroupTrans && i < NPHI) {
            const int col = 16 * tile + c16;
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) S[i][t][e] = (16 * t + 4 * g16 + e == col) ? 1.f : 0.f;
        } else if (MODE == kGroupTrans) {
#pragma unroll
            for (int t = 0; t < RT; ++t) S[i][t] = zero4();
        } else {
            if (seg == 0)   // (bad page ids are counted by the combine kernel)
                load_state_tile<DK, DV>(start_state(a, seq, h, (size_t)DK * DV, false), tile, S[i]);
            else
                load_state_c<RT>(a.seg.state + (seg_slot * H + h) * DK * DV, tile, S[i]);
        }
    }
    float dprod = 1.f;
    const uint32_t lane16 = 16u * (uint32_t)lane;
    __builtin_amdgcn_s_waitcnt(0);

    // this wave's quarter of the chunk operands: -W (waves 0, 1) or K~^T (2, 3)
    const bool loads_w = w < kGroupWaves / 2;
    const int vbase = w * PW;                                  // first vector (LDS index)
    const int vsrc = loads_w ? vbase : vbase - G::NW;          // within its region
    auto load_slice = [&](uint4 (&r)[PW], int jj) {
        const int64_t sh = (base + c0 + jj) * H + h;
        const auto rs = loads_w ? make_rsrc((const T *)a.ws.w + sh * L::w_elems, L::w_elems * sizeof(T))
                                : make_rsrc((const T *)a.ws.kt + sh * L::kt_elems, L::kt_elems * sizeof(T));
#pragma unroll
        for (int v = 0; v < PW; ++v) r[v] = buf_load16(rs, lane16, 1024u * (vsrc + v));
    };
    // per-tile U~ (not Phi tiles) and G_63 of a chunk
    struct Own {
        float gl;
        f32x4 ut[TPW - NPHI > 0 ? TPW - NPHI : 1][4];
    };
    auto load_own = [&](Own &o, int jj) {
        const int64_t sh = (base + c0 + jj) * H + h;
        o.gl = buf_load4f(make_rsrc(a.ws.g + sh * kChunk, kChunk * sizeof(float)), 0u, 4u * (kChunk - 1));
        const auto ru = make_rsrc(a.ws.ut + sh * L::ut_elems, L::ut_elems * sizeof(float));
#pragma unroll
        for (int i = NPHI; i < TPW; ++i) {
            const int ut_tile = i * kGroupWaves + w - (MODE == kGroupTrans ? DK / 16 : 0);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const uint4 x = buf_load16(ru, lane16, 1024u * (ut_tile * 4 + mt));
                o.ut[i - NPHI][mt] = f32x4{__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z),
                                           __uint_as_float(x.w)};
            }
        }
    };
    auto store_slice = [&](const uint4 (&r)[PW], int buf) {
#pragma unroll
        for (int v = 0; v < PW; ++v) ops_lds[buf][vbase + v][lane] = r[v];
    };

    auto step = [&](const Own &o, int buf, int jj) {
        const int64_t sh = (base + c0 + jj) * H + h;
        // every operand fragment of the chunk, read from LDS up front so the
        // reads' latency overlaps instead of stalling each MFMA
        uint4 wf[G::NW], kf[NV - G::NW];
#pragma unroll
        for (int v = 0; v < G::NW; ++v) wf[v] = ops_lds[buf][v][lane];
#pragma unroll
        for (int v = 0; v < NV - G::NW; ++v) kf[v] = ops_lds[buf][G::NW + v][lane];
        T sb[TPW][FS];
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int f = 0; f < FS; ++f) sb[i][f] = from_f32<T>(S[i][f >> 2][f & 3]);
        if constexpr (kHandOff) {
            const auto rs = make_rsrc((T *)a.ws.sc + sh * L::sc_elems, L::sc_elems * sizeof(T));
#pragma unroll
            for (int i = 0; i < TPW; ++i)
#pragma unroll
                for (int v = 0; v < VS; ++v)
                    buf_store16(*(const uint4 *)&sb[i][v * VEC], rs, lane16, 1024u * ((i * kGroupWaves + w) * VS + v));
        }
        // U = U~ - W S for every tile; each -W fragment read once
        f32x4 U[TPW][4];
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                if (i < NPHI) U[i][mt] = zero4();
                else U[i][mt] = o.ut[i - NPHI][mt];
            }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int v = 0; v < VS; ++v) {
                const T *fv = (const T *)&wf[mt * VS + v];
#pragma unroll
                for (int kk = 0; kk < VEC / KW; ++kk)
#pragma unroll
                    for (int i = 0; i < TPW; ++i)
                        U[i][mt] = M::mma(M::pack(&fv[kk * KW]), M::pack(&sb[i][v * VEC + kk * KW]), U[i][mt]);
            }
        T ub[TPW][FU];
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int f = 0; f < FU; ++f) ub[i][f] = from_f32<T>(U[i][f >> 2][f & 3]);
        if constexpr (kHandOff) {
            const auto rs = make_rsrc((T *)a.ws.u + sh * L::u_elems, L::u_elems * sizeof(T));
#pragma unroll
            for (int i = 0; i < TPW; ++i)
#pragma unroll
                for (int v = 0; v < VU; ++v)
                    buf_store16(*(const uint4 *)&ub[i][v * VEC], rs, lane16, 1024u * ((i * kGroupWaves + w) * VU + v));
        }
        // S = exp(G_63) S + K~^T U; each K~^T fragment read once
        const float decay = expf(o.gl);
        if constexpr (MODE == kGroupTrans) dprod *= decay;
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int t = 0; t < RT; ++t) S[i][t] = S[i][t] * decay;
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int v = 0; v < VU; ++v) {
                const T *fv = (const T *)&kf[t * VU + v];
#pragma unroll
                for (int kk = 0; kk < VEC / KW; ++kk)
#pragma unroll
                    for (int i = 0; i < TPW; ++i)
                        S[i][t] = M::mma(M::pack(&fv[kk * KW]), M::pack(&ub[i][v * VEC + kk * KW]), S[i][t]);
            }
        // Issue order in this region: this wave's LDS writes of the next
        // chunk, every fragment read, then the MFMAs with the global loads
        // (next chunk's slice and per-tile operands) one per MFMA.
        __builtin_amdgcn_sched_group_barrier(0x200, PW, 0);   // LDS writes
        __builtin_amdgcn_sched_group_barrier(0x100, NV, 0);   // LDS reads
#pragma unroll
        for (int q = 0; q < kMfmas; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
            if (q < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
        }
    };

    // ---- pipeline: operands of chunk j in LDS buffer j & 1
    uint4 rA[PW], rB[PW];
    Own oA, oB;
    load_slice(rA, 0);
    load_own(oA, 0);
    if (n > 1) {
        load_slice(rB, 1);
        load_own(oB, 1);
    }
    store_slice(rA, 0);
    __syncthreads();
    int j = 0;
    for (; j + 2 <= n; j += 2) {
        // chunk j from buffer 0; chunk j+1's operands (rB) go to buffer 1
        store_slice(rB, 1);
        load_slice(rA, min(j + 2, n - 1));
        step(oA, 0, j);
        load_own(oA, min(j + 2, n - 1));
        __syncthreads();
        // chunk j+1 from buffer 1; chunk j+2's operands (rA) go to buffer 0
        store_slice(rA, 0);
        load_slice(rB, min(j + 3, n - 1));
        step(oB, 1, j + 1);
        load_own(oB, min(j + 3, n - 1));
        __syncthreads();
    }
    if (j < n) step(oA, 0, j);

    // ---- epilogue
    if constexpr (MODE == kGroupTrans) {
        const int64_t ssh = seg_slot * H + h;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int tile = i * kGroupWaves + w;
            if (i < NPHI) {
                const int col = 16 * tile + c16;
                T *dst = (T *)a.seg.phi + ssh * DK * DK + phi_col_pos(col);
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int r = 16 * t + 4 * g16 + e;
                        dst[(size_t)r * DK] = from_f32<T>(S[i][t][e] - (r == col ? dprod : 0.f));
                    }
            } else {
                const int ut_tile = tile - DK / 16;
                float4 *dst = (float4 *)(a.seg.r + ssh * DK * DV);
#pragma unroll
                for (int t = 0; t < RT; ++t)
                    dst[(ut_tile * RT + t) * 64 + lane] = make_float4(S[i][t][0], S[i][t][1], S[i][t][2], S[i][t][3]);
            }
        }
        if (w == 0 && lane == 0) a.seg.d[ssh] = dprod;
    }
}

}  // namespace la

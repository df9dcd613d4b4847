// Workgroup forms of the chunk scan, for throughput: the chunk operands (-W
// and K~^T, 32 KB per chunk at dk = 128) are read from HBM/L2 once per
// workgroup and shared through LDS, instead of once per 16-column wave.
//
// A workgroup owns one unit of state columns:
//   kGroupTrans   (sequence, head, segment), DK + DV columns of [Phi | R]
//                 started from [I | 0]: the segment's state map;
//   kGroupReplay  (sequence, head, segment), DV columns from the segment's
//                 entering state: the state entering each chunk and U;
//   kGroupScan    (sequence, head), DV columns over the whole sequence from
//                 its starting state: the single-level scan of a batch with
//                 more column tiles than the per-tile scan keeps resident.
//                 It hands the state entering each chunk and U to the output
//                 kernel, and writes checkpoints and the final state.
// Its 4 waves own TPW tiles each (tile i of wave w is column tile
// i * 4 + w; with that striding a wave's Phi tiles are its first DK/64).
// Per chunk j, every wave
//   1. writes its quarter of chunk j+1's operands (loaded during chunk j-1)
//      into the LDS buffer (j+1) & 1 and issues the global loads of its
//      quarter of chunk j+2;
//   2. computes chunk j from buffer j & 1: each operand fragment is read from
//      LDS once and used for all TPW tiles.  In the replay and scan forms the
//      fragments are read a few ahead of the MFMAs that use them, so the LDS
//      reads of the four waves overlap the matrix work and only a short
//      window of fragments occupies registers;
//   3. meets the others at one barrier.
#pragma once
#include <type_traits>

#include "gdr_scan.h"

namespace la {

enum : int { kGroupTrans = 1, kGroupReplay = 2, kGroupScan = 3 };
constexpr int kGroupWaves = 4;

template <typename T, int DK> struct GroupOps {
    static constexpr int VEC = Vec<T>::N;
    static constexpr int VS = DK / 4 / VEC;               // -W vectors per row tile
    static constexpr int VU = kChunk / 4 / VEC;           // K~^T vectors per row tile
    static constexpr int NW = 4 * VS;                     // -W vectors per chunk
    static constexpr int NV = NW + (DK / 16) * VU;        // all vectors (1 KB each)
    static_assert(NW == (DK / 16) * VU, "operand split");
};

// Scan waves of a workgroup: the maps of a 128 x 128 state (16 column tiles
// of [Phi | R]) run on 8 waves of 2 tiles, so every wave streams its
// fragments with 2 tiles' state in registers; the other forms on 4.
template <int DK, int DV, int MODE> constexpr int group_scan_waves() {
    return (MODE == kGroupTrans && (DK / 16) % 8 == 0 && ((DK + DV) / 16) % 8 == 0) ? 8 : kGroupWaves;
}

// LDS of the output waves (OUT): the handoff of one chunk, i.e. the state
// entering it and U of every column tile in the MFMA operand order the scan
// waves hold them ([tile][vector][lane]), and a two-chunk ring of the Q and
// P fragments of the read-out (Q's row tiles, then P's; see OutFrag), which
// every output wave reads.
template <typename T, int DK, int DV> struct GroupOutLds {
    static constexpr int NT = DV / 16, VS = DK / 4 / Vec<T>::N, VU = kChunk / 4 / Vec<T>::N;
    static constexpr int NQ = 4 * VS, NQP = NQ + 4 * VU;
    uint4 sb[NT][VS][64];
    uint4 ub[NT][VU][64];
    uint4 qp[2][NQP][64];
};

template <typename T, int DK, int DV, int MODE, bool OUT = false>
__global__ __launch_bounds__((64 * group_scan_waves<DK, DV, MODE>() * (OUT ? 2 : 1))) void gdr_group_kernel(ScanArgs a) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    using G = GroupOps<T, DK>;
    constexpr int NSW = group_scan_waves<DK, DV, MODE>();                  // scan waves
    constexpr int KW = M::KW, VEC = G::VEC, VS = G::VS, VU = G::VU, NV = G::NV, PW = NV / NSW;
    constexpr int RT = DK / 16, FS = DK / 4, FU = kChunk / 4;
    constexpr int NTU = (MODE == kGroupTrans) ? (DK + DV) / 16 : DV / 16;   // tiles per unit
    constexpr int TPW = NTU / NSW;
    constexpr int NPHI = (MODE == kGroupTrans) ? DK / 16 / NSW : 0;         // Phi tiles per wave
    constexpr bool kHandOff = MODE != kGroupTrans;
    constexpr bool kScan = MODE == kGroupScan;
    static_assert(TPW * NSW == NTU && PW * NSW == NV, "tiles and operand vectors per wave");
    static_assert(MODE != kGroupTrans || NPHI * NSW == DK / 16, "Phi tiles per wave");
    static_assert(VEC == KW && sizeof(T) == 2, "streamed step: bf16 fragments, one k-step each");
    static_assert(!OUT || NSW == kGroupWaves, "output waves pair with 4 scan waves");
    constexpr int kLoads = PW + 1 + 4 * (TPW - NPHI) + (kScan ? 1 : 0);   // global loads per chunk

    __shared__ uint4 ops_lds[2][NV][64];
    // With OUT, waves NSW .. 2 NSW - 1 are output waves: wave
    // NSW + w reads out scan wave w's tiles.  Per chunk j all waves
    // pass two barriers: A_j (the scan waves have written chunk j's handoff)
    // and B_j (the output waves have read it, so chunk j+1's may be
    // written).  The output waves compute chunk j's output while the scan
    // waves run chunk j+1; the state entering each chunk and U never reach
    // HBM.
    struct NoOutLds {};
    using OL = std::conditional_t<OUT, GroupOutLds<T, DK, DV>, NoOutLds>;
    __shared__ OL hand[1];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, c16 = lane & 15;
    const int H = a.n_heads;
    // unit -> (sequence, head[, segment]); units of consecutive ids go to
    // consecutive XCDs.  The scan form takes its (sequence, head) chain in
    // the host's dispatch order (longest first).
    int seq, h, seg = 0, len, nch, c0, c1;
    int64_t base, seg_slot = 0;
    {
        const int unit = blockIdx.x;
        const int pair = kScan ? chain_of_rank(a, unit) : unit / a.max_seg;
        seg = kScan ? 0 : unit % a.max_seg;
        if (pair < 0 || pair >= a.n_seqs * H) return;
        seq = pair / H;
        h = pair % H;
        const int cu0 = a.cu[seq];
        len = a.cu[seq + 1] - cu0;
        nch = n_chunks32(len, a.C, a.cps);
        base = slot_base_dev(cu0, seq, a.C, a.cps);
        c0 = seg * a.seg_m;
        if (!kScan && c0 >= nch) return;
        c1 = kScan ? nch : min(c0 + a.seg_m, nch);
        if (!kScan) seg_slot = slot_base_dev(cu0, seq, (int64_t)a.C * a.seg_m, a.cps) + seg;
    }
    const int n = c1 - c0;

    if constexpr (OUT) {
        if (w >= NSW) {
            // Output wave.  It stages its quarter of every chunk's Q and P
            // fragments into the ring one chunk ahead, and computes
            //   O^T = scale ((S_0^T Q^T) diag(exp G) + U^T P^T)
            // for its tiles with each fragment read from LDS once for all of
            // them, in the same MFMA order as the split output kernel (so the
            // two give identical bits).
            constexpr int NQ = OL::NQ, NQP = OL::NQP, QPW = NQP / NSW;
            static_assert(QPW * NSW == NQP, "Q/P split");
            const int wo = w - NSW;
            const int64_t cu0 = a.cu[seq];
            const uint32_t l16 = 16u * (uint32_t)lane;
            auto load_qp = [&](uint4 (&r)[QPW], uint4 &eg, int jj) {
                const int64_t sh = (base + c0 + jj) * H + h;
                const auto rq = make_rsrc((const T *)a.ws.qf + sh * L::qf_elems, L::qf_elems * sizeof(T));
                const auto rp = make_rsrc((const T *)a.ws.p + sh * L::p_elems, L::p_elems * sizeof(T));
#pragma unroll
                for (int t = 0; t < QPW; ++t) {
                    const int k = wo * QPW + t;   // wave-uniform
                    r[t] = buf_load16(k < NQ ? rq : rp, l16, 1024u * (uint32_t)(k < NQ ? k : k - NQ));
                }
                // the gates of rows c, 16 + c, 32 + c, 48 + c sit together (G layout)
                eg = buf_load16(make_rsrc(a.ws.g + sh * kChunk, kChunk * sizeof(float)), 16u * (uint32_t)c16, 0u);
            };
            auto store_qp = [&](const uint4 (&r)[QPW], int buf) {
#pragma unroll
                for (int t = 0; t < QPW; ++t) hand[0].qp[buf][wo * QPW + t][lane] = r[t];
            };
            auto out_chunk = [&](const uint4 &egv, int buf, int jj) {
                int lo, hi;
                chunk_range32(c0 + jj, len, a.C, a.cps, &lo, &hi);
                __syncthreads();   // A_jj: chunk jj's handoff is complete
                T sb[TPW][FS], ub[TPW][FU];
#pragma unroll
                for (int i = 0; i < TPW; ++i) {
                    const int tile = i * NSW + wo;
#pragma unroll
                    for (int v = 0; v < VS; ++v) *(uint4 *)&sb[i][v * VEC] = hand[0].sb[tile][v][lane];
#pragma unroll
                    for (int v = 0; v < VU; ++v) *(uint4 *)&ub[i][v * VEC] = hand[0].ub[tile][v][lane];
                }
                __syncthreads();   // B_jj: the handoff may be overwritten
                const float eg[4] = {__uint_as_float(egv.x), __uint_as_float(egv.y), __uint_as_float(egv.z),
                                     __uint_as_float(egv.w)};
                T *o = (T *)a.o + ((cu0 + lo) * H + h) * DV;
                const auto ro = make_rsrc(o, head_rows_bytes<T>(hi - lo, H, DV));
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    f32x4 acc[TPW];
#pragma unroll
                    for (int i = 0; i < TPW; ++i) acc[i] = zero4();
#pragma unroll
                    for (int v = 0; v < VS; ++v) {
                        const uint4 qv = hand[0].qp[buf][mt * VS + v][lane];
#pragma unroll
                        for (int i = 0; i < TPW; ++i)
                            acc[i] = M::mma(M::pack(&sb[i][v * VEC]), M::pack((const T *)&qv), acc[i]);
                    }
                    const float e = __builtin_amdgcn_exp2f(eg[mt] * kLog2eOut);
#pragma unroll
                    for (int i = 0; i < TPW; ++i) acc[i] = acc[i] * e;
#pragma unroll
                    for (int v = 0; v < VU; ++v) {
                        const uint4 pv = hand[0].qp[buf][NQ + mt * VU + v][lane];
#pragma unroll
                        for (int i = 0; i < TPW; ++i)
                            acc[i] = M::mma(M::pack(&ub[i][v * VEC]), M::pack((const T *)&pv), acc[i]);
                    }
#pragma unroll
                    for (int i = 0; i < TPW; ++i) {
                        T out[4];
#pragma unroll
                        for (int e4 = 0; e4 < 4; ++e4) out[e4] = from_f32<T>(acc[i][e4] * a.scale);
                        const int tile = i * NSW + wo;
                        const uint32_t voff = ((uint32_t)(16 * mt + c16) * (uint32_t)(H * DV) +
                                               (uint32_t)(16 * tile + 4 * g16)) * (uint32_t)sizeof(T);
                        buf_store_4<T>(ro, voff, out);
                    }
                }
            };
            if (n > 0) {
                uint4 qA[QPW], qB[QPW], eA, eB;
                load_qp(qA, eA, 0);
                if (n > 1) load_qp(qB, eB, 1);
                store_qp(qA, 0);
                __syncthreads();   // matches the scan waves' barrier after their first operand store
                int jj = 0;
                for (; jj + 2 <= n; jj += 2) {
                    // chunk jj from ring slot 0; chunk jj+1's fragments (qB) go to slot 1
                    const uint4 e0 = eA;
                    load_qp(qA, eA, min(jj + 2, n - 1));
                    out_chunk(e0, 0, jj);
                    store_qp(qB, 1);
                    const uint4 e1 = eB;
                    load_qp(qB, eB, min(jj + 3, n - 1));
                    out_chunk(e1, 1, jj + 1);
                    store_qp(qA, 0);
                }
                if (jj < n) out_chunk(eA, 0, jj);
            }
            return;
        }
    }

    // ---- initial state of every tile
    f32x4 S[TPW][RT];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tile = i * NSW + w;
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
            // bad page ids: counted here by wave 0 of the scan form; in the
            // two-level scan the combine kernel counts them
            if (seg == 0)
                load_state_tile<DK, DV>(start_state(a, seq, h, (size_t)DK * DV, kScan && w == 0 && i == 0), tile,
                                        S[i]);
            else
                load_state_c<RT>(a.seg.state + (seg_slot * H + h) * DK * DV, tile, S[i]);
        }
    }
    float dprod = 1.f;
    const uint32_t lane16 = 16u * (uint32_t)lane;
    // checkpoints and final state (scan form): wave w's tiles, C layout
    CkptDst ck;
    ChunkCursor cur{0, a.C, len, a.C};
    if constexpr (kScan) ck.init(a, seq, h, len, (size_t)DK * DV, w == 0);
    auto lane_off = [&](int i) {
        return 4u * (uint32_t)(4 * g16 * DV + 16 * (i * NSW + w) + c16);
    };
    auto store_state = [&](float *d) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) store_state_tiles<RT, DV>(d, S[i], lane_off(i));
    };
    __builtin_amdgcn_s_waitcnt(0);

    // this wave's quarter of the chunk operands: -W (waves 0, 1) or K~^T (2, 3)
    const bool loads_w = w < NSW / 2;
    const int vbase = w * PW;                                  // first vector (LDS index)
    const int vsrc = loads_w ? vbase : vbase - G::NW;          // within its region
    auto load_slice = [&](uint4 (&r)[PW], int jj) {
        const int64_t sh = (base + c0 + jj) * H + h;
        const auto rs = loads_w ? make_rsrc((const T *)a.ws.w + sh * L::w_elems, L::w_elems * sizeof(T))
                                : make_rsrc((const T *)a.ws.kt + sh * L::kt_elems, L::kt_elems * sizeof(T));
#pragma unroll
        for (int v = 0; v < PW; ++v) r[v] = buf_load16(rs, lane16, 1024u * (vsrc + v));
    };
    // per-tile U~ (not Phi tiles), G_63 of a chunk and, in the scan form, the
    // page id of the checkpoint the chunk would end
    struct Own {
        float gl;
        int ckid;
        f32x4 ut[TPW - NPHI > 0 ? TPW - NPHI : 1][4];
    };
    auto load_own = [&](Own &o, int jj) {
        const int64_t sh = (base + c0 + jj) * H + h;
        o.gl = buf_load4f(make_rsrc(a.ws.g + sh * kChunk, kChunk * sizeof(float)), 0u, 4u * (kChunk - 1));
        o.ckid = kScan ? ck.load_id(jj / a.cps) : 0;
        const auto ru = make_rsrc((const T *)a.ws.ut + sh * L::ut_elems, L::ut_elems * sizeof(T));
#pragma unroll
        for (int i = NPHI; i < TPW; ++i) {
            const int ut_tile = i * NSW + w - (MODE == kGroupTrans ? DK / 16 : 0);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) o.ut[i - NPHI][mt] = load_ut<T>(ru, (uint32_t)lane, (uint32_t)(ut_tile * 4 + mt));
        }
    };
    auto store_slice = [&](const uint4 (&r)[PW], int buf) {
#pragma unroll
        for (int v = 0; v < PW; ++v) ops_lds[buf][vbase + v][lane] = r[v];
    };

    // Streamed step: the chunk's NV fragments are read from LDS kAhead
    // ahead of the TPW MFMAs each feeds.  The U phase walks the -W
    // fragments dk-step-major (fragment f = 4 v + mt is row tile mt, dk step
    // v), so the state's bf16 operand of dk step v is formed just before its
    // four fragments; every accumulator still sums its dk steps in order, as
    // in the whole-chunk form.
    auto step_stream = [&](const Own &o, int buf, int jj) {
        typedef T tx8 __attribute__((ext_vector_type(8)));
        constexpr int kAhead = 4;
        const int64_t sh = (base + c0 + jj) * H + h;
        auto lds_vec = [](int f) { return f < G::NW ? (f & 3) * VS + (f >> 2) : f; };
        uint4 fr[NV];
#pragma unroll
        for (int f = 0; f < kAhead; ++f) fr[f] = ops_lds[buf][lds_vec(f)][lane];
        f32x4 U[TPW][4];
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) U[i][mt] = i < NPHI ? zero4() : o.ut[i - NPHI][mt];   // Phi tiles take no U~
        const auto rsc = make_rsrc((T *)a.ws.sc + sh * L::sc_elems, L::sc_elems * sizeof(T));
#pragma unroll
        for (int v = 0; v < VS; ++v) {
            tx8 sv[TPW];
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
#pragma unroll
                for (int e = 0; e < 8; ++e) sv[i][e] = from_f32<T>(S[i][2 * v + (e >> 2)][e & 3]);
                if constexpr (OUT)
                    hand[0].sb[i * NSW + w][v][lane] = __builtin_bit_cast(uint4, sv[i]);
                else if constexpr (kHandOff)
                    buf_store16(__builtin_bit_cast(uint4, sv[i]), rsc, lane16,
                                1024u * ((i * NSW + w) * VS + v));
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int f = 4 * v + mt;
                if (f + kAhead < NV) fr[f + kAhead] = ops_lds[buf][lds_vec(f + kAhead)][lane];
                const tx8 av = __builtin_bit_cast(tx8, fr[f]);
#pragma unroll
                for (int i = 0; i < TPW; ++i) U[i][mt] = M::mma(av, sv[i], U[i][mt]);
            }
        }
        tx8 ub[TPW][VU];
        const auto ru = make_rsrc((T *)a.ws.u + sh * L::u_elems, L::u_elems * sizeof(T));
#pragma unroll
        for (int i = 0; i < TPW; ++i)
#pragma unroll
            for (int v = 0; v < VU; ++v) {
#pragma unroll
                for (int e = 0; e < 8; ++e) ub[i][v][e] = from_f32<T>(U[i][2 * v + (e >> 2)][e & 3]);
                if constexpr (OUT)
                    hand[0].ub[i * NSW + w][v][lane] = __builtin_bit_cast(uint4, ub[i][v]);
                else if constexpr (kHandOff)
                    buf_store16(__builtin_bit_cast(uint4, ub[i][v]), ru, lane16,
                                1024u * ((i * NSW + w) * VU + v));
            }
        // S = exp(G_63) S + K~^T U
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
                const int f = G::NW + t * VU + v;
                if (f + kAhead < NV) fr[f + kAhead] = ops_lds[buf][lds_vec(f + kAhead)][lane];
                const tx8 av = __builtin_bit_cast(tx8, fr[f]);
#pragma unroll
                for (int i = 0; i < TPW; ++i) S[i][t] = M::mma(av, ub[i][v], S[i][t]);
            }
        // Issue order in this region: this wave's LDS writes of the next
        // chunk, the first kAhead fragment reads, then per fragment one more
        // read and its TPW MFMAs, the global loads (next chunk's slice and
        // per-tile operands) one per MFMA.
        __builtin_amdgcn_sched_group_barrier(0x200, PW, 0);       // LDS writes
        __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);   // LDS reads
        int q = 0;
#pragma unroll
        for (int f = 0; f < NV; ++f) {
            if (f + kAhead < NV) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
            for (int i = 0; i < TPW; ++i, ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
                if (q < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
            }
        }
    };
    auto step = [&](const Own &o, int buf, int jj) { step_stream(o, buf, jj); };
    // After chunk jj's barrier (scan form): its checkpoint, if it ends on a
    // multiple of C.  S still holds the state after chunk jj.
    auto after = [&](int ckid) {
        if constexpr (kScan) {
            if (cur.advance()) {
                if (float *d = ck.next(ckid)) store_state(d);
            }
        }
    };

    // ---- pipeline: operands of chunk j in LDS buffer j & 1
    if (n > 0) {
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
            const int id0 = oA.ckid;
            load_own(oA, min(j + 2, n - 1));
            __syncthreads();                        // (with OUT: A_j)
            if constexpr (OUT) __syncthreads();     // B_j
            after(id0);
            // chunk j+1 from buffer 1; chunk j+2's operands (rA) go to buffer 0
            store_slice(rA, 0);
            load_slice(rB, min(j + 3, n - 1));
            step(oB, 1, j + 1);
            const int id1 = oB.ckid;
            load_own(oB, min(j + 3, n - 1));
            __syncthreads();
            if constexpr (OUT) __syncthreads();
            after(id1);
        }
        if (j < n) {
            step(oA, 0, j);
            if constexpr (OUT) {   // the output waves wait on the last chunk's handoff
                __syncthreads();
                __syncthreads();
            }
            after(oA.ckid);
        }
    }

    // ---- epilogue
    if constexpr (kScan) {
        if (a.final_state) store_state(a.final_state + (size_t)(seq * H + h) * DK * DV);
    }
    if constexpr (MODE == kGroupTrans) {
        const int64_t ssh = seg_slot * H + h;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int tile = i * NSW + w;
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

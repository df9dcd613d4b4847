// Scan with output wave over two column tiles (bf16): the per-tile scan of
// gdr_scan1o_kernel with one workgroup per (sequence, head, pair of 16-column
// tiles).  The scan wave keeps both tiles' state (all DK rows) in registers;
// every -W and K~^T fragment it loads feeds both tiles' MFMAs, and the
// output wave's Q and P fragments feed both tiles' read-outs.  Per tile the
// MFMAs, their operands and their order are those of the one-tile kernel, so
// the two give identical bits.  A CU that holds several scan workgroups of a
// large batch moves half the operand bytes per tile through its load path,
// which bounds those workgroups' chunk steps; a batch whose one-tile
// workgroups all fit at once keeps the one-tile kernel, whose chain step is
// shorter (half the MFMAs per chunk).
#pragma once
#include "gdr_scan.h"

namespace la {

constexpr int kPairTiles = 2;

template <typename T, int DK, int DV>
__device__ inline void scan2_chunks(const ScanArgs &a, int seq, int h, int tp, int len, int64_t base, int nch,
                                    f32x4 (&S)[kPairTiles][DK / 16], Handoff<T, DK> *hs) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    constexpr int KW = M::KW, VEC = Vec<T>::N, P = kPairTiles;
    constexpr int RT = DK / 16, FS = DK / 4, FU = kChunk / 4;
    constexpr int VS = FS / VEC, VU = FU / VEC;
    constexpr int kMfmas = P * (4 * (FS / KW) + RT * (FU / KW));   // per chunk
    constexpr int kLoads = 1 + 4 * P + 4 * VS + RT * VU;            // operand loads per chunk

    const int lane = threadIdx.x & 63, g16 = lane >> 4, c16 = lane & 15;
    const int H = a.n_heads;
    ChunkCursor cur{0, a.C, len, a.C};
    CkptDst ck;
    ck.init(a, seq, h, len, (size_t)DK * DV, tp == 0);
    uint32_t lane_off[P];
#pragma unroll
    for (int i = 0; i < P; ++i) lane_off[i] = 4u * (uint32_t)(4 * g16 * DV + 16 * (P * tp + i) + c16);
    __builtin_amdgcn_s_waitcnt(0);

    struct Ops {
        float gl;
        int ckid;
        f32x4 ut[P][4];
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
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) o.ut[i][mt] = load_ut<T>(ru, (uint32_t)lane, (uint32_t)((P * tp + i) * 4 + mt));
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
        T sb[P][FS];
#pragma unroll
        for (int i = 0; i < P; ++i) {
#pragma unroll
            for (int f = 0; f < FS; ++f) sb[i][f] = from_f32<T>(S[i][f >> 2][f & 3]);
#pragma unroll
            for (int v = 0; v < VS; ++v) hs[i].sb[jj & 1][v][lane] = *(const uint4 *)&sb[i][v * VEC];
        }
        f32x4 U[P][4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const T *wv = (const T *)&o.wn[mt][0];
#pragma unroll
            for (int i = 0; i < P; ++i) U[i][mt] = o.ut[i][mt];
#pragma unroll
            for (int ks = 0; ks < FS / KW; ++ks)
#pragma unroll
                for (int i = 0; i < P; ++i)
                    U[i][mt] = M::mma(M::pack(&wv[ks * KW]), M::pack(&sb[i][ks * KW]), U[i][mt]);
        }
        T ub[P][FU];
#pragma unroll
        for (int i = 0; i < P; ++i) {
#pragma unroll
            for (int f = 0; f < FU; ++f) ub[i][f] = from_f32<T>(U[i][f >> 2][f & 3]);
#pragma unroll
            for (int v = 0; v < VU; ++v) hs[i].ub[jj & 1][v][lane] = *(const uint4 *)&ub[i][v * VEC];
        }
        const float decay = expf(o.gl);
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            const T *kv = (const T *)&o.kt[t][0];
#pragma unroll
            for (int i = 0; i < P; ++i) S[i][t] = S[i][t] * decay;
#pragma unroll
            for (int ks = 0; ks < FU / KW; ++ks)
#pragma unroll
                for (int i = 0; i < P; ++i) S[i][t] = M::mma(M::pack(&kv[ks * KW]), M::pack(&ub[i][ks * KW]), S[i][t]);
        }
        // the next chunk's loads interleaved one per MFMA (see scan1_chunks)
#pragma unroll
        for (int i = 0; i < kMfmas; ++i) {
            if (i < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
        }
        if (cur.advance()) {
            if (float *d = ck.next(o.ckid)) {
#pragma unroll
                for (int i = 0; i < P; ++i) store_state_tiles<RT, DV>(d, S[i], lane_off[i]);
            }
        }
        lds_barrier();   // this chunk's slots are written; the output wave may read them
    };
    scan_ring<1>(nch, load, step, (Ops *)nullptr);
}

// The output wave: per chunk, after the scan wave's barrier, the read-out of
// both tiles from one set of Q and P fragments (loaded one chunk ahead).
template <typename T, int DK, int DV>
__device__ inline void out_wave2_chunks(const ScanArgs &a, int h, int tp, int64_t cu0, int len, int64_t base,
                                        int nch, const Handoff<T, DK> *hs) {
    using F = OutFrag<T, DK>;
    constexpr int VEC = Vec<T>::N, VS = Handoff<T, DK>::VS, VU = Handoff<T, DK>::VU, P = kPairTiles;
    const int lane = threadIdx.x & 63, H = a.n_heads;
    ChunkCursor cur{0, a.C, len, a.C};
    auto load = [&](F &f, int jj) { load_out_frag<T, DK>(f, a.ws, (base + jj) * H + h); };
    auto step = [&](const F &f, int jj) {
        const int lo = cur.pos;
        cur.advance();
        const int n = cur.pos - lo;
        lds_barrier();
#pragma unroll
        for (int i = 0; i < P; ++i) {
            T sb[VS * VEC], ub[VU * VEC];
#pragma unroll
            for (int v = 0; v < VS; ++v) *(uint4 *)&sb[v * VEC] = hs[i].sb[jj & 1][v][lane];
#pragma unroll
            for (int v = 0; v < VU; ++v) *(uint4 *)&ub[v * VEC] = hs[i].ub[jj & 1][v][lane];
            out_tile<T, DK>(f, sb, ub, a.scale, (T *)a.o + ((cu0 + lo) * H + h) * DV, n, H, DV, P * tp + i);
        }
    };
    scan_ring<1>(nch, load, step, (F *)nullptr);
}

template <typename T, int DK, int DV>
__global__ __launch_bounds__(128) void gdr_scan2o_kernel(ScanArgs a) {
    static_assert(sizeof(T) == 2, "bf16 operands");
    constexpr int NP = DV / 16 / kPairTiles;   // workgroups per (sequence, head)
    __shared__ Handoff<T, DK> hs[kPairTiles];
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = chain_of_rank(a, xcd + 8 * (q / NP)), tp = q % NP;
    const int H = a.n_heads;
    if (pair < 0) return;
    const int seq = pair / H, h = pair % H;
    const int cu0 = a.cu[seq], len = a.cu[seq + 1] - cu0;
    const int nch = n_chunks32(len, a.C, a.cps);
    const int64_t base = slot_base_dev(cu0, seq, a.C, a.cps);
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    if (wave == 0) {
        f32x4 S[kPairTiles][DK / 16];
        const float *src = start_state(a, seq, h, (size_t)DK * DV, tp == 0);
#pragma unroll
        for (int i = 0; i < kPairTiles; ++i) load_state_tile<DK, DV>(src, kPairTiles * tp + i, S[i]);
        scan2_chunks<T, DK, DV>(a, seq, h, tp, len, base, nch, S, hs);
        if (a.final_state) {
            const int lane = threadIdx.x & 63;
#pragma unroll
            for (int i = 0; i < kPairTiles; ++i)
                store_state_tiles<DK / 16, DV>(a.final_state + (size_t)pair * DK * DV, S[i],
                                               4u * (uint32_t)(4 * (lane >> 4) * DV + 16 * (kPairTiles * tp + i) + (lane & 15)));
        }
    } else {
        out_wave2_chunks<T, DK, DV>(a, h, tp, cu0, len, base, nch, hs);
    }
}

}  // namespace la

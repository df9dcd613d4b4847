// Inter-chunk scan: the sequential part of the prefill.  One wave owns the
// state columns [tile*BV, (tile+1)*BV) of one (sequence, head); those columns
// evolve independently of the others.  Per chunk, with S the fp32 state
// entering it (kept in MFMA accumulator registers for the whole sequence):
//   U       = U~ - W S                  (64 x BV, bf16/fp32 MFMA, fp32 accumulate)
//   S_next  = exp(G_63) S + K~^T U      (DK x BV)
// The state enters both products straight from its accumulator layout; the
// -W and K~^T operands were written by the preparation kernel with the
// matching contraction permutation, so no lane shuffles or LDS are needed.
// The wave also hands the output kernel the state entering each chunk and U
// (both in the io type), and writes fp32 checkpoints and the final state.
#pragma once
#include "la_common.h"

namespace la {

struct ScanArgs {
    const int32_t *cu;
    const float *state_in;        // [n_seqs, H, DK, DV] or null (zero state)
    float *final_state;           // [n_seqs, H, DK, DV] or null
    float *ckpt;                  // [rows, H, DK, DV] or null
    const int32_t *ckpt_off;      // [n_seqs]
    int32_t n_seqs, n_heads, C, cps;
    Workspace ws;
};

template <typename T, int DK, int DV, int BV>
__global__ __launch_bounds__(64) void gdr_scan_kernel(ScanArgs a) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    constexpr int KW = M::KW, VEC = Vec<T>::N;
    constexpr int RT = DK / 16;          // state row tiles
    constexpr int CT = BV / 16;          // state column tiles owned by this wave
    constexpr int NT = DV / BV;          // waves per (sequence, head)
    constexpr int FS = DK / 4;           // per-lane operand values over dk
    constexpr int FU = kChunk / 4;       // per-lane operand values over chunk rows
    static_assert(FS % VEC == 0 && FU % VEC == 0, "vector width");

    const int lane = threadIdx.x, g16 = lane >> 4, c16 = lane & 15;
    // XCD-aware unit mapping: workgroups are dealt to the 8 XCDs round-robin,
    // so keep the NT tiles of one (sequence, head) on one XCD, where they
    // share the chunk operands through that XCD's L2.
    const int b = blockIdx.x, xcd = b & 7, q = b >> 3;
    const int pair = xcd + 8 * (q / NT), tile = q % NT;
    const int H = a.n_heads;
    if (pair >= a.n_seqs * H) return;
    const int seq = pair / H, h = pair % H;
    const int64_t cu0 = a.cu[seq], len = (int64_t)a.cu[seq + 1] - cu0;
    const int64_t nch = n_chunks(len, a.C, a.cps);
    const int64_t base = slot_base(cu0, seq, a.C, a.cps);
    const size_t state_off = (size_t)pair * DK * DV;

    f32x4 S[RT][CT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = 16 * rt + 4 * g16 + i, col = tile * BV + 16 * ct + c16;
                S[rt][ct][i] = a.state_in ? a.state_in[state_off + (size_t)row * DV + col] : 0.f;
            }

    for (int64_t j = 0; j < nch; ++j) {
        const int64_t sh = (base + j) * H + h;
        // chunk operands
        T wn[4][FS];
        T kt[RT][FU];
        {
            const uint4 *src = (const uint4 *)((const T *)a.ws.w + sh * L::w_elems);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int v = 0; v < FS / VEC; ++v)
                    *(uint4 *)&wn[mt][v * VEC] = src[(mt * (FS / VEC) + v) * 64 + lane];
            const uint4 *srk = (const uint4 *)((const T *)a.ws.kt + sh * L::kt_elems);
#pragma unroll
            for (int mt = 0; mt < RT; ++mt)
#pragma unroll
                for (int v = 0; v < FU / VEC; ++v)
                    *(uint4 *)&kt[mt][v * VEC] = srk[(mt * (FU / VEC) + v) * 64 + lane];
        }
        f32x4 U[4][CT];
        {
            const float4 *ut = (const float4 *)(a.ws.ut + sh * L::ut_elems);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    const float4 x = ut[((tile * CT + ct) * 4 + mt) * 64 + lane];
                    U[mt][ct] = f32x4{x.x, x.y, x.z, x.w};
                }
        }
        const float decay = expf(a.ws.g[sh * kChunk + kChunk - 1]);

        // state entering the chunk, as B operand over dk (io type)
        T sb[CT][FS];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int f = 0; f < FS; ++f) sb[ct][f] = from_f32<T>(S[f >> 2][ct][f & 3]);
        {
            uint4 *dst = (uint4 *)((T *)a.ws.sc + sh * L::sc_elems);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int v = 0; v < FS / VEC; ++v)
                    dst[((tile * CT + ct) * (FS / VEC) + v) * 64 + lane] = *(const uint4 *)&sb[ct][v * VEC];
        }
        // U = U~ + (-W) S
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int ks = 0; ks < FS / KW; ++ks)
                    U[mt][ct] = M::mma(M::pack(&wn[mt][ks * KW]), M::pack(&sb[ct][ks * KW]), U[mt][ct]);
        // U as B operand over chunk rows
        T ub[CT][FU];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int f = 0; f < FU; ++f) ub[ct][f] = from_f32<T>(U[f >> 2][ct][f & 3]);
        {
            uint4 *dst = (uint4 *)((T *)a.ws.u + sh * L::u_elems);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int v = 0; v < FU / VEC; ++v)
                    dst[((tile * CT + ct) * (FU / VEC) + v) * 64 + lane] = *(const uint4 *)&ub[ct][v * VEC];
        }
        // S = exp(G_63) S + K~^T U
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                f32x4 acc = S[rt][ct] * decay;
#pragma unroll
                for (int ks = 0; ks < FU / KW; ++ks)
                    acc = M::mma(M::pack(&kt[rt][ks * KW]), M::pack(&ub[ct][ks * KW]), acc);
                S[rt][ct] = acc;
            }
        // checkpoint when the chunk ends on a multiple of C
        if (a.ckpt) {
            int64_t lo, hi;
            chunk_range(j, len, a.C, a.cps, &lo, &hi);
            if (hi % a.C == 0) {
                const int64_t row = (int64_t)a.ckpt_off[seq] + hi / a.C - 1;
                float *dst = a.ckpt + ((size_t)row * H + h) * DK * DV;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            dst[(size_t)(16 * rt + 4 * g16 + i) * DV + tile * BV + 16 * ct + c16] =
                                S[rt][ct][i];
            }
        }
    }
    if (a.final_state) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    a.final_state[state_off + (size_t)(16 * rt + 4 * g16 + i) * DV + tile * BV +
                                  16 * ct + c16] = S[rt][ct][i];
    }
}

}  // namespace la

// Output read-out: parallel over (chunk, head, sequence), 4 waves each.
// For chunk rows r, with S_0 the state entering the chunk and U from the
// scan:
//   o_r = scale * ( exp(G_r) (S_0^T q_r) + sum_{s<=r} exp(G_r - G_s) (q_r . k_s) u_s )
// i.e. O = scale * ( diag(exp G) Q S_0 + (Q K^T  masked r>=s, decayed) U ),
// the read-out of the post-update state S_r^T q_r.
#pragma once
#include "la_common.h"

namespace la {

constexpr float kLog2eOut = 1.4426950408889634f;

struct OutArgs {
    const void *q, *k;
    void *o;
    const int32_t *cu;
    int32_t n_seqs, n_heads, C, cps, max_chunks;
    float scale;
    Workspace ws;
};

template <typename T, int DK, int DV> struct alignas(16) OutSmem {
    static constexpr int PK = Vec<T>::N;
    T qs[kChunk][DK + PK];
    T ks[kChunk][DK + PK];
    T ps[kChunk][kChunk + PK];        // decayed, masked Q K^T
    T os[kChunk][DV + PK];            // output staging for coalesced stores
    float G[kChunk];                  // log2(e)-scaled cumulative gate
};

template <typename T, int DK, int DV>
__global__ __launch_bounds__(256, 2) void gdr_out_kernel(OutArgs a) {
    using M = MT<T>;
    using L = WsLayout<T, DK, DV>;
    constexpr int KW = M::KW, KSTEP = M::KSTEP, VEC = Vec<T>::N;
    constexpr int FS = DK / 4, FU = kChunk / 4;
    constexpr int NTW = DV / 16 / 4;  // output column tiles per wave
    static_assert(NTW >= 1, "dv >= 64");
    __shared__ OutSmem<T, DK, DV> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g16 = lane >> 4, c16 = lane & 15;
    int64_t j;
    int seq, h;
    if (!unit_of_block(a.n_seqs, a.n_heads, a.max_chunks, &seq, &h, &j)) return;
    const int H = a.n_heads;
    const int64_t cu0 = a.cu[seq];
    const int len = a.cu[seq + 1] - a.cu[seq];
    if (j >= n_chunks32(len, a.C, a.cps)) return;
    int lo, hi;
    chunk_range32((int)j, len, a.C, a.cps, &lo, &hi);
    const int n = hi - lo;
    const int64_t t0 = cu0 + lo;
    const int64_t sh = (slot_base(cu0, seq, a.C, a.cps) + j) * H + h;

    // state entering the chunk and U for this wave's column tiles (issued
    // first, so their latency overlaps the Q and K staging loads)
    T sc[NTW][FS], ub[NTW][FU];
    {
        const T *scsrc = (const T *)a.ws.sc + sh * L::sc_elems;
        const T *usrc = (const T *)a.ws.u + sh * L::u_elems;
#pragma unroll
        for (int w = 0; w < NTW; ++w) {
            const int nt = wave * NTW + w;
#pragma unroll
            for (int v = 0; v < FS / VEC; ++v)
                *(uint4 *)&sc[w][v * VEC] = ((const uint4 *)scsrc)[(nt * (FS / VEC) + v) * 64 + lane];
#pragma unroll
            for (int v = 0; v < FU / VEC; ++v)
                *(uint4 *)&ub[w][v * VEC] = ((const uint4 *)usrc)[(nt * (FU / VEC) + v) * 64 + lane];
        }
    }
    const T *qin = (const T *)a.q;
    const T *kin = (const T *)a.k;
    {
        // all loads in flight before the first LDS store; rows past the end
        // read the last valid row and are zeroed
        constexpr int IT = kChunk * DK / VEC / 256;
        static_assert(IT * 256 * VEC == kChunk * DK, "tiling");
        uint4 qv[IT], kv[IT];
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            const int rr = r < n ? r : n - 1;
            qv[it] = *(const uint4 *)(qin + ((t0 + rr) * H + h) * DK + c);
            kv[it] = *(const uint4 *)(kin + ((t0 + rr) * H + h) * DK + c);
        }
        const float gl = tid < kChunk ? a.ws.g[sh * kChunk + tid] : 0.f;
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            if (r >= n) {
                qv[it] = make_uint4(0, 0, 0, 0);
                kv[it] = make_uint4(0, 0, 0, 0);
            }
            *(uint4 *)&sm.qs[r][c] = qv[it];
            *(uint4 *)&sm.ks[r][c] = kv[it];
        }
        if (tid < kChunk) sm.G[tid] = gl * kLog2eOut;
    }
    __syncthreads();

    // log2(e)-scaled cumulative gates this lane needs, read once
    float grow[4][4], gcol[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) grow[mt][i] = sm.G[16 * mt + 4 * g16 + i];
        gcol[mt] = sm.G[16 * mt + c16];
    }

    // P = (Q K^T) * exp(G_r - G_s) on r >= s, zero above the diagonal
    {
        const int mt = wave;     // run-time row tile: its gates come from LDS
        const float4 gw4 = *(const float4 *)&sm.G[16 * mt + 4 * g16];
        const float gw[4] = {gw4.x, gw4.y, gw4.z, gw4.w};
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            f32x4 acc = zero4();
            if (nt <= mt) {
#pragma unroll
                for (int ks = 0; ks < DK / KSTEP; ++ks)
                    acc = M::mma(M::pack(&sm.qs[16 * mt + c16][ks * KSTEP + g16 * KW]),
                                 M::pack(&sm.ks[16 * nt + c16][ks * KSTEP + g16 * KW]), acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * g16 + i, s = 16 * nt + c16;
                const float e = __builtin_amdgcn_exp2f(gw[i] - gcol[nt]);
                sm.ps[r][s] = from_f32<T>((s <= r) ? acc[i] * e : 0.f);
            }
        }
    }
    __syncthreads();

#pragma unroll
    for (int w = 0; w < NTW; ++w) {
        const int nt = wave * NTW + w;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int r = 16 * mt + c16;
            f32x4 acc = zero4();
            // Q S_0 (contraction over dk in the state's permuted order)
#pragma unroll
            for (int ks = 0; ks < FS / KW; ++ks) {
                const int f0 = ks * KW;
                const typename M::frag fa =
                    M::pack2(&sm.qs[r][perm_row(f0, g16)], &sm.qs[r][perm_row(f0 + (KW > 4 ? 4 : 0), g16)]);
                acc = M::mma(fa, M::pack(&sc[w][f0]), acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] *= __builtin_amdgcn_exp2f(grow[mt][i]);
            // + P U (contraction over chunk rows in U's permuted order)
#pragma unroll
            for (int ks = 0; ks < FU / KW; ++ks) {
                const int f0 = ks * KW;
                const typename M::frag fa =
                    M::pack2(&sm.ps[r][perm_row(f0, g16)], &sm.ps[r][perm_row(f0 + (KW > 4 ? 4 : 0), g16)]);
                acc = M::mma(fa, M::pack(&ub[w][f0]), acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                sm.os[16 * mt + 4 * g16 + i][16 * nt + c16] = from_f32<T>(acc[i] * a.scale);
        }
    }
    __syncthreads();
    T *oout = (T *)a.o;
    for (int vi = tid; vi < kChunk * DV / VEC; vi += 256) {
        const int r = vi / (DV / VEC), c = (vi % (DV / VEC)) * VEC;
        if (r < n) *(uint4 *)(oout + ((t0 + r) * H + h) * DV + c) = *(const uint4 *)&sm.os[r][c];
    }
}

}  // namespace la

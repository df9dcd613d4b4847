// Chunk preparation: everything about a chunk that does not depend on the
// state entering it.  One workgroup (4 waves) per (chunk, head, sequence).
//
// For chunk rows r, s = 0..63 (rows past the chunk's end are zero-padded,
// which makes them inert: zero key, zero value, zero beta, zero gate):
//   G_r   = sum_{s<=r} g_s                      (chunk-local, fp32)
//   Gp_r  = G_{r-1} (literal rule; G_{-1} = 0) or G_r (decayed rule)
//   A     = strictly lower part of beta_r exp(Gp_r - G_s) (k_r . k_s)
//   X     = (I + A)^{-1}                       (unit lower triangular, fp32)
//   W     = X diag(beta exp(Gp)) K             (stored negated, A-operand order;
//                                               computed as W^T tiles, whose
//                                               accumulator layout is that order)
//   U~    = X diag(beta) V                     (fp32, C-layout)
//   K~^T  = (diag(exp(G_63 - G)) K)^T          (A-operand order, chunk rows permuted)
//   P     = (Q K^T) exp(G_r - G_s) on s <= r   (for the output; B operand of P^T
//                                               per token tile, chunk rows permuted)
//   Q     = the queries as the B operand of Q^T per token tile (dk permuted)
// so that, for the state S_0 entering the chunk, U = U~ - W S_0 holds the
// per-row corrections u_r = beta_r (v_r - pred_r) and the state leaving the
// chunk is exp(G_63) S_0 + K~^T U.  (Derivation: unroll the recurrence
// inside the chunk; the prediction of row r sees S_0 decayed by exp(Gp_r)
// plus the rank-one writes of earlier rows decayed by exp(Gp_r - G_s).)
//
// K and V are staged row-major only; operands that contract over chunk rows
// are read with the LDS transpose read (bf16) or one element per lane (fp32).
// Exponentials of gate differences use exp2 on log2(e)-scaled cumulative
// gates; every exponent is a difference formed before exponentiation.
#pragma once
#include "la_common.h"

namespace la {

struct PrepArgs {
    const void *q, *k, *v;
    const float *g, *beta;
    const int32_t *cu;
    int32_t n_seqs, n_heads, C, cps, variant, max_chunks;
    Workspace ws;
    int32_t chunk_major;   // block map (see unit_of_block)
};

constexpr float kLog2e = 1.4426950408889634f;

// Cross-lane moves (DPP): CTRL selects the source lane, ROWS enables rows of
// 16 lanes; lanes without a source, and disabled rows, read 0.
template <int CTRL, int ROWS = 0xF>
__device__ inline float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWS, 0xF, true));
}

// Inclusive prefix sum over the wave's 64 lanes: shifts within each row of
// 16 lanes, then each row's carry from the rows before it (row broadcasts).
__device__ inline float wave_inclusive_sum(float x) {
    x += dpp_f<0x111>(x);          // row_shr:1
    x += dpp_f<0x112>(x);          // row_shr:2
    x += dpp_f<0x114>(x);          // row_shr:4
    x += dpp_f<0x118>(x);          // row_shr:8
    x += dpp_f<0x142, 0xA>(x);     // row_bcast:15 into rows 1 and 3
    x += dpp_f<0x143, 0xC>(x);     // row_bcast:31 into rows 2 and 3
    return x;
}

// One column-oriented step of the diagonal-block substitution: lane s of
// each row holds the final x[s] of its columns; broadcast it along the row
// (row_newbcast:s) and subtract L[r][s] x[s] (L is zero at and above the
// diagonal, so rows r <= s are left unchanged).
template <int S>
__device__ inline void subst_step(float (&x)[4], const float (&L)[16]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) x[c] -= L[S] * dpp_f<0x150 + S>(x[c]);
}

template <int S = 0>
__device__ inline void subst_all(float (&x)[4], const float (&L)[16]) {
    if constexpr (S < 16) {
        subst_step<S>(x, L);
        subst_all<S + 1>(x, L);
    }
}

template <typename T, int DK, int DV> struct alignas(16) PrepSmem {
    static constexpr int PK = Vec<T>::N;       // row pads keep 16-byte alignment
    static constexpr int DM = DK > DV ? DK : DV;
    T ks[kChunk][DK + PK];                     // K, row-major
    T vs[kChunk][DM + PK];                     // V, row-major
    float am[kChunk][kChunk + 4];              // A (strictly lower)
    float xm[kChunk][kChunk + 4];              // X = (I + A)^{-1}
    float ysc[4][16][17];                      // per-wave 16x16 scratch
    float G2[kChunk], Gp2[kChunk], bs[kChunk]; // log2e-scaled gates, beta
    float dW[kChunk], dK[kChunk];              // beta exp(Gp), exp(G_63 - G)
};

// 16x16x16 fp32 product of two LDS blocks with fp32 MFMA, accumulated in c.
__device__ inline f32x4 mm16_f32(const float *A, int lda, const float *B, int ldb, f32x4 c,
                                 int lane) {
    const int r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(A[r * lda + 4 * ks + g], B[(4 * ks + g) * ldb + r],
                                                 c, 0, 0, 0);
    return c;
}

// Operands that contract over the rows of a row-major LDS tile.
template <typename T> struct RowTile;

template <> struct RowTile<__bf16> {
    typedef short i16x4 __attribute__((ext_vector_type(4)));
    // LDS transpose read: in each 16-lane group, source lane s reads 4
    // elements of row `row(s)` at column n0 + 4 (s % 4); with row(s) chosen
    // as base + s / 4, lane i of the group receives column n0 + i of rows
    // base .. base + 3.
    __device__ static inline i16x4 tr4(const __bf16 *tile, int ld, int row, int n0, int lane) {
        const int s = lane & 15;
        const __bf16 *p = tile + row * ld + n0 + 4 * (s & 3);
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)p);
    }
    // B operand (32 x 16, natural k order): rows [k0, k0 + 32), columns [n0, n0 + 16)
    __device__ static inline bf16x8 bfrag(const __bf16 *tile, int ld, int k0, int n0, int lane) {
        const int g = lane >> 4, s = lane & 15;
        const i16x4 lo = tr4(tile, ld, k0 + 8 * g + (s >> 2), n0, lane);
        const i16x4 hi = tr4(tile, ld, k0 + 8 * g + 4 + (s >> 2), n0, lane);
        typedef short i16x8 __attribute__((ext_vector_type(8)));
        const i16x8 both = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, both);
    }
    // tile[perm_row(f, g)][n0 + lane % 16] for f = 4q .. 4q + 3
    __device__ static inline void col4(const __bf16 *tile, int ld, int q, int n0, int lane, float *out) {
        const int g = lane >> 4, s = lane & 15;
        const i16x4 v = tr4(tile, ld, 16 * q + 4 * g + (s >> 2), n0, lane);
#pragma unroll
        for (int t = 0; t < 4; ++t) out[t] = (float)__builtin_bit_cast(__bf16, (short)v[t]);
    }
};

template <> struct RowTile<float> {
    // B operand (4 x 16): one element per lane
    __device__ static inline float bfrag(const float *tile, int ld, int k0, int n0, int lane) {
        return tile[(k0 + (lane >> 4)) * ld + n0 + (lane & 15)];
    }
    __device__ static inline void col4(const float *tile, int ld, int q, int n0, int lane, float *out) {
        const int g = lane >> 4;
#pragma unroll
        for (int t = 0; t < 4; ++t) out[t] = tile[(16 * q + 4 * g + t) * ld + n0 + (lane & 15)];
    }
};

// Two workgroups per CU where the LDS allows (fp32 operands with a
// 128-wide head dimension need more than half of it).
template <typename T, int DK, int DV>
__global__ __launch_bounds__(256, sizeof(PrepSmem<T, DK, DV>) <= 80 * 1024 ? 2 : 1) void gdr_prep_kernel(PrepArgs a) {
    using M = MT<T>;
    using RT = RowTile<T>;
    using Sm = PrepSmem<T, DK, DV>;
    constexpr int KW = M::KW, KSTEP = M::KSTEP, VEC = Vec<T>::N;
    constexpr int LDK = DK + Sm::PK, LDV = Sm::DM + Sm::PK, LDA = kChunk + 4;
    __shared__ Sm sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g16 = lane >> 4, c16 = lane & 15;
    int64_t j;
    int seq, h;
    if (!unit_of_block(a.n_seqs, a.n_heads, a.max_chunks, a.chunk_major != 0, &seq, &h, &j)) return;
    const int H = a.n_heads;
    const int64_t cu0 = a.cu[seq];
    const int len = a.cu[seq + 1] - a.cu[seq];
    if (j >= n_chunks32(len, a.C, a.cps)) return;
    int lo, hi;
    chunk_range32((int)j, len, a.C, a.cps, &lo, &hi);
    const int n = hi - lo;
    const int64_t t0 = cu0 + lo;
    const int64_t sh = (slot_base_dev(cu0, seq, a.C, a.cps) + j) * H + h;   // slot-head index

    const T *kin = (const T *)a.k;
    const T *vin = (const T *)a.v;

    // This lane's queries: token row 16 wave + lane % 16 at dk perm_row(f, g)
    // for f < DK/4 (g = lane / 16), runs of 4.  That is exactly this lane's
    // part of the B operand of Q^T for token tile `wave` in the order the
    // state's accumulator layout contracts dk, so it is stored as is for the
    // output, and the P product below contracts dk in the same order.
    T qf[DK / 4];
    {
        const int r = 16 * wave + c16, rr = r < n ? r : n - 1;
        const T *qrow = (const T *)a.q + ((t0 + rr) * H + h) * DK + 4 * g16;
#pragma unroll
        for (int p4 = 0; p4 < DK / 16; ++p4) {
            if constexpr (sizeof(T) == 2)
                *(uint2 *)&qf[4 * p4] = *(const uint2 *)(qrow + 16 * p4);
            else
                *(uint4 *)&qf[4 * p4] = *(const uint4 *)(qrow + 16 * p4);
        }
    }

    // ---- 1. stage K, V (row-major), g, beta; clear X ------------------------
    // Every global load is issued before the first use; rows past the
    // chunk's end read the last valid row and are zeroed afterwards.
    {
        constexpr int KIT = kChunk * DK / VEC / 256, VIT = kChunk * DV / VEC / 256;
        static_assert(KIT * 256 * VEC == kChunk * DK && VIT * 256 * VEC == kChunk * DV, "tiling");
        uint4 kr[KIT], vr[VIT];
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            const int rr = r < n ? r : n - 1;
            kr[it] = *(const uint4 *)(kin + ((t0 + rr) * H + h) * DK + c);
        }
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DV / VEC), c = (vi % (DV / VEC)) * VEC;
            const int rr = r < n ? r : n - 1;
            vr[it] = *(const uint4 *)(vin + ((t0 + rr) * H + h) * DV + c);
        }
        float gv = 0.f, bv = 0.f;
        if (tid < kChunk) {
            const int rr = tid < n ? tid : n - 1;
            gv = a.g[(t0 + rr) * H + h];
            bv = a.beta[(t0 + rr) * H + h];
        }
        for (int e = tid; e < kChunk * LDA; e += 256) (&sm.xm[0][0])[e] = 0.f;
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            if (r >= n) kr[it] = make_uint4(0, 0, 0, 0);
            *(uint4 *)&sm.ks[r][c] = kr[it];
        }
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DV / VEC), c = (vi % (DV / VEC)) * VEC;
            if (r >= n) vr[it] = make_uint4(0, 0, 0, 0);
            *(uint4 *)&sm.vs[r][c] = vr[it];
        }
        // ---- 2. chunk-local gate prefix sum (wave 0) --------------------------
        if (wave == 0) {
            const float b = tid < n ? bv : 0.f;
            const float x = wave_inclusive_sum(tid < n ? gv : 0.f);
            const float prev = dpp_f<0x138>(x);   // wave_shr:1: lane - 1's sum, 0 on lane 0
            const float gp = (a.variant == 0) ? prev : x;
            const float g63 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
            sm.G2[lane] = x * kLog2e;
            sm.Gp2[lane] = gp * kLog2e;
            sm.bs[lane] = b;
            sm.dW[lane] = b * __builtin_amdgcn_exp2f(gp * kLog2e);
            sm.dK[lane] = __builtin_amdgcn_exp2f((g63 - x) * kLog2e);
            a.ws.g[sh * kChunk + 4 * (lane & 15) + (lane >> 4)] = x;   // G layout: row 16 m + c at 4 c + m
        }
    }
    __syncthreads();

    // ---- 3. A = strictly-lower beta_r exp(Gp_r - G_s) K K^T ------------------
    // Wave w computes row tile w against all four column tiles: four
    // independent MFMA chains with no branch between them (the tiles above
    // the diagonal are computed and dropped: they are never read).  The row
    // tile's K fragments are read once and reused for every column tile.
    {
        const int mt = wave;
        typename M::frag ka[DK / KSTEP];
#pragma unroll
        for (int ks = 0; ks < DK / KSTEP; ++ks) ka[ks] = M::pack(&sm.ks[16 * mt + c16][ks * KSTEP + g16 * KW]);
        f32x4 acc[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            acc[nt] = zero4();
#pragma unroll
            for (int ks = 0; ks < DK / KSTEP; ++ks)
                acc[nt] = M::mma(ka[ks], M::pack(&sm.ks[16 * nt + c16][ks * KSTEP + g16 * KW]), acc[nt]);
        }
        const float4 brow = *(const float4 *)&sm.bs[16 * mt + 4 * g16];
        const float4 gprow = *(const float4 *)&sm.Gp2[16 * mt + 4 * g16];
        const float bv[4] = {brow.x, brow.y, brow.z, brow.w};
        const float gv[4] = {gprow.x, gprow.y, gprow.z, gprow.w};
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            if (nt > mt) continue;   // wave-uniform
            const float gcol = sm.G2[16 * nt + c16];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * g16 + i, s = 16 * nt + c16;
                const float e = __builtin_amdgcn_exp2f(gv[i] - gcol);
                sm.am[r][s] = (s < r) ? bv[i] * e * acc[nt][i] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- 4. X = (I + A)^{-1}: diagonal 16-blocks by substitution ---------------
    // Wave w inverts block w with all 64 lanes: lane (q, r), q = lane / 16,
    // r = lane % 16, holds row r of columns 4q .. 4q + 3 of the block's
    // inverse.  Each x[r] receives the updates L[r][s] x[s] in the order
    // s = 0, 1, ..., as forward substitution does.
    {
        const int base = 16 * wave, q = lane >> 4, r = lane & 15;
        float L[16];
#pragma unroll
        for (int s4 = 0; s4 < 16; s4 += 4) {
            const float4 v = *(const float4 *)&sm.am[base + r][base + s4];
            L[s4] = v.x;
            L[s4 + 1] = v.y;
            L[s4 + 2] = v.z;
            L[s4 + 3] = v.w;
        }
        float x[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) x[c] = (r == 4 * q + c) ? 1.f : 0.f;
        subst_all(x, L);
        *(float4 *)&sm.xm[base + r][base + 4 * q] = make_float4(x[0], x[1], x[2], x[3]);
    }
    __syncthreads();
    // off-diagonal blocks by bands: X_ij = -X_ii sum_{k=j}^{i-1} A_ik X_kj
    for (int d = 1; d < 4; ++d) {
        const int bi = d + wave, bj = wave;
        const bool active = bi < 4;
        if (active) {
            f32x4 y = zero4();
            for (int bk = bj; bk < bi; ++bk)
                y = mm16_f32(&sm.am[16 * bi][16 * bk], LDA, &sm.xm[16 * bk][16 * bj], LDA, y, lane);
#pragma unroll
            for (int i = 0; i < 4; ++i) sm.ysc[wave][4 * g16 + i][c16] = y[i];
        }
        // ysc[wave] is written and read by this wave alone: its LDS accesses
        // execute in order, so only the compiler needs holding back here
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (active) {
            f32x4 xij = mm16_f32(&sm.xm[16 * bi][16 * bi], LDA, &sm.ysc[wave][0][0], 17, zero4(), lane);
#pragma unroll
            for (int i = 0; i < 4; ++i) sm.xm[16 * bi + 4 * g16 + i][16 * bj + c16] = -xij[i];
        }
        __syncthreads();
    }

    // ---- 5. W, U~ = X diag(beta) V, K~^T, P and Q fragments --------------------
    {
        const int mt = wave;
        constexpr int NKS = kChunk / KSTEP;
        typename M::frag f1[NKS], f2[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            T v1[KW], v2[KW];
#pragma unroll
            for (int jj = 0; jj < KW; ++jj) {
                const int s = ks * KSTEP + g16 * KW + jj;
                const float x = sm.xm[16 * mt + c16][s];
                v1[jj] = from_f32<T>(x * sm.dW[s]);
                v2[jj] = from_f32<T>(x * sm.bs[s]);
            }
            f1[ks] = M::pack(v1);
            f2[ks] = M::pack(v2);
        }
        // W^T tile (dk tile nt, row tile mt) = K^T (X diag(dW))^T: per lane the
        // K fragment read as a B operand of K is the A operand of K^T, and f1
        // (A operand of X diag(dW)) is the B operand of its transpose.  The
        // accumulator then holds W[16 mt + c16][16 nt + 4 g + i], element
        // 4 nt + i of this lane's -W fragment in the scan's permuted dk
        // order, so -W is stored straight from registers.
        {
            T wf[DK / 4];
#pragma unroll
            for (int nt = 0; nt < DK / 16; ++nt) {
                f32x4 acc = zero4();
#pragma unroll
                for (int ks = 0; ks < NKS; ++ks)
                    acc = M::mma(RT::bfrag(&sm.ks[0][0], LDK, ks * KSTEP, 16 * nt, lane), f1[ks], acc);
#pragma unroll
                for (int i = 0; i < 4; ++i) wf[4 * nt + i] = from_f32<T>(-acc[i]);
            }
            constexpr int NV = DK / 4 / VEC;
            T *wout = (T *)a.ws.w + sh * WsLayout<T, DK, DV>::w_elems;
#pragma unroll
            for (int v = 0; v < NV; ++v)
                *(uint4 *)(wout + ((size_t)(mt * NV + v) * 64 + lane) * VEC) = *(const uint4 *)&wf[v * VEC];
        }
        T *ut = (T *)a.ws.ut + sh * WsLayout<T, DK, DV>::ut_elems;
#pragma unroll
        for (int nt = 0; nt < DV / 16; ++nt) {
            f32x4 acc = zero4();
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
                acc = M::mma(f2[ks], RT::bfrag(&sm.vs[0][0], LDV, ks * KSTEP, 16 * nt, lane), acc);
            T u4[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) u4[i] = from_f32<T>(acc[i]);
            if constexpr (sizeof(T) == 4)
                *(uint4 *)(ut + ((size_t)(nt * 4 + mt) * 64 + lane) * 4) = *(const uint4 *)u4;
            else
                *(uint2 *)(ut + ((size_t)(nt * 4 + mt) * 64 + lane) * 4) = *(const uint2 *)u4;
        }
        // K~^T: per dk row tile, lane holds 16 values at chunk rows perm_row(f, g)
        T *kout = (T *)a.ws.kt + sh * WsLayout<T, DK, DV>::kt_elems;
        constexpr int NV2 = 16 / VEC;
        for (int kt = wave; kt < DK / 16; kt += 4) {
            T vals[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float c4[4];
                RT::col4(&sm.ks[0][0], LDK, q, 16 * kt, lane, c4);
                const float4 d = *(const float4 *)&sm.dK[16 * q + 4 * g16];
                vals[4 * q + 0] = from_f32<T>(c4[0] * d.x);
                vals[4 * q + 1] = from_f32<T>(c4[1] * d.y);
                vals[4 * q + 2] = from_f32<T>(c4[2] * d.z);
                vals[4 * q + 3] = from_f32<T>(c4[3] * d.w);
            }
#pragma unroll
            for (int v = 0; v < NV2; ++v)
                *(uint4 *)(kout + ((size_t)(kt * NV2 + v) * 64 + lane) * VEC) = *(const uint4 *)&vals[v * VEC];
        }
        // P for token tile mt, computed as the tiles K Q^T: the result tile
        // (s tile nt, token tile mt) holds P[16 mt + c16][16 nt + 4 g + i] in
        // lane (g, c16), which is element 4 nt + i of that lane's P^T
        // operand, so the fragments are stored straight from the
        // accumulators.  Tiles above the diagonal are zero.
        {
            const float gr = sm.G2[16 * mt + c16];
            T vals[16];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                f32x4 acc = zero4();
                if (nt <= mt) {
#pragma unroll
                    for (int ks = 0; ks < DK / KSTEP; ++ks) {
                        const int f0 = ks * KW;
                        const T *krow = &sm.ks[16 * nt + c16][0];
                        acc = M::mma(M::pack2(krow + perm_row(f0, g16), krow + perm_row(f0 + (KW > 4 ? 4 : 0), g16)),
                                     M::pack(&qf[f0]), acc);
                    }
                }
                const float4 gs = *(const float4 *)&sm.G2[16 * nt + 4 * g16];
                const float gsv[4] = {gs.x, gs.y, gs.z, gs.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int s = 16 * nt + 4 * g16 + i, r = 16 * mt + c16;
                    const float e = __builtin_amdgcn_exp2f(gr - gsv[i]);
                    vals[4 * nt + i] = from_f32<T>(s <= r ? acc[i] * e : 0.f);
                }
            }
            T *pout = (T *)a.ws.p + sh * WsLayout<T, DK, DV>::p_elems;
#pragma unroll
            for (int v = 0; v < NV2; ++v)
                *(uint4 *)(pout + ((size_t)(mt * NV2 + v) * 64 + lane) * VEC) = *(const uint4 *)&vals[v * VEC];
            constexpr int NQ = DK / 4 / VEC;
            T *qout = (T *)a.ws.qf + sh * WsLayout<T, DK, DV>::qf_elems;
#pragma unroll
            for (int v = 0; v < NQ; ++v)
                *(uint4 *)(qout + ((size_t)(mt * NQ + v) * 64 + lane) * VEC) = *(const uint4 *)&qf[v * VEC];
        }
    }
}

}  // namespace la

// Chunk preparation: everything about a chunk that does not depend on the
// state entering it.  One workgroup (4 waves) per (chunk, head, sequence).
//
// For chunk rows r, s = 0..63 (rows past the chunk's end are zero-padded,
// which makes them inert: zero key, zero value, zero beta, zero gate):
//   G_r   = sum_{s<=r} g_s                      (chunk-local, fp32)
//   Gp_r  = G_{r-1} (literal rule; G_{-1} = 0) or G_r (decayed rule)
//   A     = strictly lower part of beta_r exp(Gp_r - G_s) (k_r . k_s)
//   X     = (I + A)^{-1}                       (unit lower triangular, fp32)
//   W     = X diag(beta exp(Gp)) K             (stored negated, A-operand order)
//   U~    = X diag(beta) V                     (fp32, C-layout)
//   K~^T  = (diag(exp(G_63 - G)) K)^T          (A-operand order, chunk rows permuted)
// so that, for the state S_0 entering the chunk, U = U~ - W S_0 holds the
// per-row corrections u_r = beta_r (v_r - pred_r) and the state leaving the
// chunk is exp(G_63) S_0 + K~^T U.  (Derivation: unroll the recurrence
// inside the chunk; the prediction of row r sees S_0 decayed by exp(Gp_r)
// plus the rank-one writes of earlier rows decayed by exp(Gp_r - G_s).)
#pragma once
#include "la_common.h"

namespace la {

struct PrepArgs {
    const void *k, *v;
    const float *g, *beta;
    const int32_t *cu;
    int32_t n_heads, C, cps, variant;
    Workspace ws;
};

template <typename T, int DK, int DV> struct PrepSmem {
    static constexpr int PK = Vec<T>::N;      // row pads keep 16-byte alignment
    T ks[kChunk][DK + PK];                    // K, row-major
    T kst[DK][kChunk + PK];                   // K^T
    T vst[DV][kChunk + PK];                   // V^T
    float am[kChunk][kChunk + 1];             // A (strictly lower)
    float xm[kChunk][kChunk + 1];             // X = (I + A)^{-1}
    float ysc[4][16][17];                     // per-wave 16x16 scratch
    float gs[kChunk], bs[kChunk], G[kChunk], Gp[kChunk];
    float dW[kChunk], dK[kChunk];             // beta exp(Gp), exp(G_63 - G)
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

template <typename T, int DK, int DV>
__global__ __launch_bounds__(256) void gdr_prep_kernel(PrepArgs a) {
    using M = MT<T>;
    constexpr int KW = M::KW, KSTEP = M::KSTEP, VEC = Vec<T>::N;
    __shared__ PrepSmem<T, DK, DV> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g16 = lane >> 4, c16 = lane & 15;
    const int64_t j = blockIdx.x;
    const int h = blockIdx.y, seq = blockIdx.z, H = a.n_heads;
    const int64_t cu0 = a.cu[seq], len = (int64_t)a.cu[seq + 1] - cu0;
    if (j >= n_chunks(len, a.C, a.cps)) return;
    int64_t lo, hi;
    chunk_range(j, len, a.C, a.cps, &lo, &hi);
    const int n = (int)(hi - lo);
    const int64_t t0 = cu0 + lo;
    const int64_t sh = (slot_base(cu0, seq, a.C, a.cps) + j) * H + h;   // slot-head index

    const T *kin = (const T *)a.k;
    const T *vin = (const T *)a.v;

    // ---- 1. stage K, K^T, V^T, g, beta in LDS; clear X -----------------------
    for (int vi = tid; vi < kChunk * DK / VEC; vi += 256) {
        const int r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
        T buf[VEC];
        if (r < n) {
            const uint4 raw = *(const uint4 *)(kin + ((t0 + r) * H + h) * DK + c);
            *(uint4 *)buf = raw;
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) buf[e] = from_f32<T>(0.f);
        }
        *(uint4 *)&sm.ks[r][c] = *(const uint4 *)buf;
#pragma unroll
        for (int e = 0; e < VEC; ++e) sm.kst[c + e][r] = buf[e];
    }
    for (int vi = tid; vi < kChunk * DV / VEC; vi += 256) {
        const int r = vi / (DV / VEC), c = (vi % (DV / VEC)) * VEC;
        T buf[VEC];
        if (r < n) {
            *(uint4 *)buf = *(const uint4 *)(vin + ((t0 + r) * H + h) * DV + c);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) buf[e] = from_f32<T>(0.f);
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) sm.vst[c + e][r] = buf[e];
    }
    if (tid < kChunk) {
        const bool ok = tid < n;
        sm.gs[tid] = ok ? a.g[(t0 + tid) * H + h] : 0.f;
        sm.bs[tid] = ok ? a.beta[(t0 + tid) * H + h] : 0.f;
    }
    for (int e = tid; e < kChunk * (kChunk + 1); e += 256) (&sm.xm[0][0])[e] = 0.f;
    __syncthreads();

    // ---- 2. chunk-local gate prefix sum (wave 0) ------------------------------
    if (wave == 0) {
        float x = sm.gs[lane];
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const float y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        const float prev = __shfl_up(x, 1, 64);
        const float gp = (a.variant == 0) ? (lane == 0 ? 0.f : prev) : x;
        const float g63 = __shfl(x, 63, 64);
        sm.G[lane] = x;
        sm.Gp[lane] = gp;
        sm.dW[lane] = sm.bs[lane] * expf(gp);
        sm.dK[lane] = expf(g63 - x);
        a.ws.g[sh * kChunk + lane] = x;
    }
    __syncthreads();

    // ---- 3. A = strictly-lower beta_r exp(Gp_r - G_s) K K^T ------------------
    {
        const int mt = wave;
        for (int nt = 0; nt <= mt; ++nt) {
            f32x4 acc = zero4();
#pragma unroll
            for (int ks = 0; ks < DK / KSTEP; ++ks) {
                const typename M::frag fa = M::pack(&sm.ks[16 * mt + c16][ks * KSTEP + g16 * KW]);
                const typename M::frag fb = M::pack(&sm.ks[16 * nt + c16][ks * KSTEP + g16 * KW]);
                acc = M::mma(fa, fb, acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * g16 + i, s = 16 * nt + c16;
                sm.am[r][s] = (s < r) ? sm.bs[r] * expf(sm.Gp[r] - sm.G[s]) * acc[i] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- 4. X = (I + A)^{-1}: diagonal 16-blocks by substitution ---------------
    if (lane < 16) {
        const int base = 16 * wave;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float acc = (r == lane) ? 1.f : 0.f;
#pragma unroll
            for (int s = 0; s < r; ++s) acc -= sm.am[base + r][base + s] * x[s];
            x[r] = acc;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) sm.xm[base + r][base + lane] = x[r];
    }
    __syncthreads();
    // off-diagonal blocks by bands: X_ij = -X_ii sum_{k=j}^{i-1} A_ik X_kj
    for (int d = 1; d < 4; ++d) {
        const int bi = d + wave, bj = wave;
        const bool active = bi < 4;
        if (active) {
            f32x4 y = zero4();
            for (int bk = bj; bk < bi; ++bk)
                y = mm16_f32(&sm.am[16 * bi][16 * bk], kChunk + 1, &sm.xm[16 * bk][16 * bj],
                             kChunk + 1, y, lane);
#pragma unroll
            for (int i = 0; i < 4; ++i) sm.ysc[wave][4 * g16 + i][c16] = y[i];
        }
        __syncthreads();
        if (active) {
            f32x4 xij = mm16_f32(&sm.xm[16 * bi][16 * bi], kChunk + 1, &sm.ysc[wave][0][0], 17,
                                 zero4(), lane);
#pragma unroll
            for (int i = 0; i < 4; ++i) sm.xm[16 * bi + 4 * g16 + i][16 * bj + c16] = -xij[i];
        }
        __syncthreads();
    }

    // ---- 5. W = X diag(dW) K (staged in ks), U~ = X diag(beta) V (to workspace) --
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
        f32x4 wt[DK / 16];
#pragma unroll
        for (int nt = 0; nt < DK / 16; ++nt) {
            f32x4 acc = zero4();
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
                acc = M::mma(f1[ks], M::pack(&sm.kst[16 * nt + c16][ks * KSTEP + g16 * KW]), acc);
            wt[nt] = acc;
        }
        float4 *ut = (float4 *)(a.ws.ut + sh * WsLayout<T, DK, DV>::ut_elems);
#pragma unroll
        for (int nt = 0; nt < DV / 16; ++nt) {
            f32x4 acc = zero4();
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
                acc = M::mma(f2[ks], M::pack(&sm.vst[16 * nt + c16][ks * KSTEP + g16 * KW]), acc);
            ut[(nt * 4 + mt) * 64 + lane] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        }
        __syncthreads();   // every wave is done reading ks (step 3) before it is overwritten
#pragma unroll
        for (int nt = 0; nt < DK / 16; ++nt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                sm.ks[16 * mt + 4 * g16 + i][16 * nt + c16] = from_f32<T>(-wt[nt][i]);
    }
    __syncthreads();

    // ---- 6. write -W and K~^T in A-operand order -------------------------------
    {
        // -W: per row tile mt, lane: DK/4 values at columns perm_row(f, g)
        constexpr int NV = DK / 4 / VEC;
        T *wout = (T *)a.ws.w + sh * WsLayout<T, DK, DV>::w_elems;
        for (int vi = tid; vi < 4 * NV * 64; vi += 256) {
            const int ln = vi & 63, v = (vi >> 6) % NV, mt = vi / (64 * NV);
            const int r = 16 * mt + (ln & 15), g = ln >> 4;
            T buf[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) buf[e] = sm.ks[r][perm_row(v * VEC + e, g)];
            *(uint4 *)(wout + (size_t)vi * VEC) = *(const uint4 *)buf;
        }
        // K~^T: per dk row tile mt, lane: 16 values at chunk rows perm_row(f, g)
        constexpr int NV2 = 16 / VEC;
        T *kout = (T *)a.ws.kt + sh * WsLayout<T, DK, DV>::kt_elems;
        for (int vi = tid; vi < (DK / 16) * NV2 * 64; vi += 256) {
            const int ln = vi & 63, v = (vi >> 6) % NV2, mt = vi / (64 * NV2);
            const int m = 16 * mt + (ln & 15), g = ln >> 4;
            T buf[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int s = perm_row(v * VEC + e, g);
                buf[e] = from_f32<T>(sm.dK[s] * to_f32(sm.kst[m][s]));
            }
            *(uint4 *)(kout + (size_t)vi * VEC) = *(const uint4 *)buf;
        }
    }
}

}  // namespace la

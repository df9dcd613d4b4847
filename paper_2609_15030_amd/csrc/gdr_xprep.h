// Chunk preparation for the fused scan (bf16 operands): the part of a chunk
// that depends on its keys and gates only.  One workgroup (4 waves) per
// (chunk, head, sequence).
//
// For chunk rows r, s = 0..63 (rows past the chunk's end are zero-padded:
// zero key, zero beta, zero gate, so they are inert):
//   G_r  = sum_{s<=r} g_s                     (chunk-local)
//   Gp_r = G_{r-1} (literal rule; G_{-1} = 0) or G_r (decayed rule)
//   A    = strictly lower part of beta_r exp(Gp_r - G_s) (k_r . k_s)
//   X    = (I + A)^{-1}                      (unit lower triangular, fp32)
// With S_0 the state entering the chunk, the corrections
//   U = X diag(beta) (V - diag(exp(Gp)) K S_0)
// hold u_r = beta_r (v_r - pred_r): unrolling the recurrence inside the
// chunk, the prediction of row r sees S_0 decayed by exp(Gp_r) plus the
// rank-one writes of the earlier rows s decayed by exp(Gp_r - G_s).  The
// scan evaluates that product itself; this kernel writes what it needs that
// the inputs do not hold:
//   X diag(beta) in bf16 as MFMA A-operand fragments whose columns are permuted the way
//     the scan holds the rows of its C-layout accumulators (perm_row): row
//     tile mt, k-step ks, lane (g, c): X[16 mt + c][perm_row(8 ks + j, g)],
//     j < 8.  X is lower triangular, so only k-steps ks <= mt / 2 are stored
//     (6 fragments of 1 KB: slot xfrag_slot(mt, ks));
//   the gate block: G, exp(Gp), beta and exp(G_63 - G), 64 fp32 each.
// Both sit in one 7 KB block per chunk-head (X fragments, then the gate
// block), which the scan copies into LDS as is.
// Every exponent is a difference formed before exponentiation (<= 0 when
// g <= 0): no exp(-G) factor is ever formed.
#pragma once
#include "gdr_prep.h"   // DPP scan, substitution and fp32 block product helpers

namespace la {

constexpr int kXFrags = 6;                     // stored X fragments per chunk-head
constexpr int kGateBlock = 4 * kChunk;         // floats of the gate block per chunk-head
constexpr int kMiscVec = kXFrags * 64 + kGateBlock / 4;   // 16-byte vectors per chunk-head block (7 KB)

__device__ __host__ inline int xfrag_slot(int mt, int ks) { return mt < 2 ? mt : 2 * mt - 2 + ks; }

struct XPrepArgs {
    const void *k;
    const float *g, *beta;
    const int32_t *cu;
    int32_t n_seqs, n_heads, C, cps, variant, max_chunks;
    uint4 *misc;       // per slot-head: X diag(beta) fragments [kXFrags][64 lanes] x 16 B,
                       // then the gate block [4][64] fp32: G, exp(Gp), beta, exp(G_63 - G)
    int32_t chunk_major;
};

// A and X are unit-lower-triangular: only their ten 16x16 blocks (bi, bj),
// bj <= bi, are stored, each with a 17-float row pitch (a column read by
// the fp32 products touches 16 distinct banks).
constexpr int kTriBlocks = 10, kBlkPitch = 17, kBlkFloats = 16 * kBlkPitch;
__device__ inline int tri_blk(int bi, int bj) { return bi * (bi + 1) / 2 + bj; }

template <int DK> struct alignas(16) XPrepSmem {
    static constexpr int LDK = DK + 8;          // bf16 row pitch (16-byte aligned rows)
    // K (staged row-major, read by the A = K K^T products) is dead once those
    // products are in registers; the blocks of A and X take its place.  The
    // small footprint lets seven workgroups share a CU.
    union {
        __bf16 ks[kChunk][LDK];
        struct {
            float a[kTriBlocks * kBlkFloats];   // A (strictly lower)
            float x[kTriBlocks * kBlkFloats];   // X = (I + A)^{-1}
        } t;
    };
    float G2[kChunk], Gp2[kChunk], bs[kChunk];  // log2e-scaled gates, beta
    __device__ float *ablk(int bi, int bj) { return t.a + tri_blk(bi, bj) * kBlkFloats; }
    __device__ float *xblk(int bi, int bj) { return t.x + tri_blk(bi, bj) * kBlkFloats; }
};

template <int DK>
__global__ __launch_bounds__(256) void gdr_xprep_kernel(XPrepArgs a) {
    using M = MT<__bf16>;
    using Sm = XPrepSmem<DK>;
    constexpr int KW = M::KW, KSTEP = M::KSTEP, LB = kBlkPitch;
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
    const __bf16 *kin = (const __bf16 *)a.k;

    // ---- 1. stage K (row-major), g, beta ----------------------------------
    // Rows past the chunk's end read the last valid row and are zeroed.
    {
        constexpr int VEC = 8, KIT = kChunk * DK / VEC / 256;
        static_assert(KIT * 256 * VEC == kChunk * DK, "tiling");
        uint4 kr[KIT];
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            const int rr = r < n ? r : n - 1;
            kr[it] = *(const uint4 *)(kin + ((t0 + rr) * H + h) * DK + c);
        }
        float gv = 0.f, bv = 0.f;
        if (tid < kChunk) {
            const int rr = tid < n ? tid : n - 1;
            gv = a.g[(t0 + rr) * H + h];
            bv = a.beta[(t0 + rr) * H + h];
        }
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const int vi = tid + 256 * it, r = vi / (DK / VEC), c = (vi % (DK / VEC)) * VEC;
            if (r >= n) kr[it] = make_uint4(0, 0, 0, 0);
            *(uint4 *)&sm.ks[r][c] = kr[it];
        }
        // ---- 2. chunk-local gate prefix sum (wave 0); the gate block --------
        if (wave == 0) {
            const float b = tid < n ? bv : 0.f;
            const float x = wave_inclusive_sum(tid < n ? gv : 0.f);
            const float prev = dpp_f<0x138>(x);   // wave_shr:1: lane - 1's sum, 0 on lane 0
            const float gp = (a.variant == 0) ? prev : x;
            const float g63 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
            sm.G2[lane] = x * kLog2e;
            sm.Gp2[lane] = gp * kLog2e;
            sm.bs[lane] = b;
            float *gb = (float *)(a.misc + sh * kMiscVec + kXFrags * 64);
            gb[lane] = x;
            gb[kChunk + lane] = __builtin_amdgcn_exp2f(gp * kLog2e);
            gb[2 * kChunk + lane] = b;
            gb[3 * kChunk + lane] = __builtin_amdgcn_exp2f((g63 - x) * kLog2e);
        }
    }
    __syncthreads();

    // ---- 3. A = strictly-lower beta_r exp(Gp_r - G_s) K K^T -----------------
    // Wave w computes row tile w against all four column tiles (tiles above
    // the diagonal are computed and dropped).  The row tile's K fragments are
    // read once and reused for every column tile.
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
        float gcol[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) gcol[nt] = sm.G2[16 * nt + c16];
        __syncthreads();   // every wave's K reads are done: A takes K's LDS
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            if (nt > mt) continue;   // wave-uniform
            float *ab = sm.ablk(mt, nt);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 16 * mt + 4 * g16 + i, s = 16 * nt + c16;
                const float e = __builtin_amdgcn_exp2f(gv[i] - gcol[nt]);
                ab[(4 * g16 + i) * LB + c16] = (s < r) ? bv[i] * e * acc[nt][i] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- 4. X = (I + A)^{-1}: diagonal 16-blocks by substitution -------------
    // Wave w inverts block w with all 64 lanes: lane (q, r), q = lane / 16,
    // r = lane % 16, holds row r of columns 4q .. 4q + 3 of the block's
    // inverse.  Each x[r] receives the updates L[r][s] x[s] in the order
    // s = 0, 1, ..., as forward substitution does.
    {
        const int q = lane >> 4, r = lane & 15;
        const float *ab = sm.ablk(wave, wave);
        float L[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) L[s] = ab[r * LB + s];
        float x[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) x[c] = (r == 4 * q + c) ? 1.f : 0.f;
        subst_all(x, L);
        float *xb = sm.xblk(wave, wave);
#pragma unroll
        for (int c = 0; c < 4; ++c) xb[r * LB + 4 * q + c] = x[c];
    }
    __syncthreads();
    // off-diagonal blocks by bands: X_ij = -X_ii sum_{k=j}^{i-1} A_ik X_kj.
    // The sum goes through block X_ij itself, which no other wave reads in
    // this band: the wave writes it, reads it back as the B operand of the
    // product with X_ii, and overwrites it with the result.
    for (int d = 1; d < 4; ++d) {
        const int bi = d + wave, bj = wave;
        const bool active = bi < 4;
        float *xij_blk = active ? sm.xblk(bi, bj) : nullptr;
        if (active) {
            f32x4 y = zero4();
            for (int bk = bj; bk < bi; ++bk) y = mm16_f32(sm.ablk(bi, bk), LB, sm.xblk(bk, bj), LB, y, lane);
#pragma unroll
            for (int i = 0; i < 4; ++i) xij_blk[(4 * g16 + i) * LB + c16] = y[i];
        }
        // the block is written and read by this wave alone: its LDS accesses
        // execute in order, so only the compiler needs holding back here
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (active) {
            f32x4 xij = mm16_f32(sm.xblk(bi, bi), LB, xij_blk, LB, zero4(), lane);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int i = 0; i < 4; ++i) xij_blk[(4 * g16 + i) * LB + c16] = -xij[i];
        }
        __syncthreads();
    }

    // ---- 5. X fragments: row tile mt = wave, k-steps ks <= mt / 2 -------------
    // Lane (g, c) takes row r = 16 mt + c at columns perm_row(8 ks + j, g):
    // two runs of 4, at 16 (2 ks) + 4 g and 16 (2 ks + 1) + 4 g.  Entries
    // above the diagonal are zero (blocks above it are not stored).
    {
        const int mt = wave, r = 16 * mt + c16;
        uint4 *xout = a.misc + sh * kMiscVec;
        for (int ks = 0; ks <= (mt >> 1); ++ks) {
            __bf16 v8[8];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int bc = 2 * ks + half, s0 = 16 * bc + 4 * g16;
                const float *xb = bc <= mt ? sm.xblk(mt, bc) : nullptr;   // wave-uniform
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v8[4 * half + e] = (__bf16)(xb && s0 + e <= r ? xb[c16 * LB + 4 * g16 + e] * sm.bs[s0 + e] : 0.f);
            }
            xout[xfrag_slot(mt, ks) * 64 + lane] = *(const uint4 *)v8;
        }
    }
}

}  // namespace la

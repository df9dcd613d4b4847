// Fused chunk scan (bf16 operands): the sequential recurrence and the output
// read-out, with every chunk's keys, queries and values staged once per
// workgroup in LDS.
//
// A workgroup owns CW state columns of one (sequence, head) and runs its
// chunks in order; its CW / 32 waves own 32 columns (two 16-column tiles)
// each and keep them in fp32 MFMA result registers (C layout: lane (g, c)
// holds rows 4 g + i of every 16-row tile, column c).  Per chunk, with S_0
// the state entering it and the gate block and X written by the
// preparation kernel (gdr_xprep.h):
//
//   Y  = K S_0                           A = K rows, B = S_0 (k = dk, perm_row)
//   Z  = diag(beta) V - diag(d) Y        d = beta exp(Gp), V read in C layout
//   U  = X Z                             A = X fragments, B = Z (k = chunk rows)
//   S_1 = exp(G_63) S_0 + K^T diag(exp(G_63 - G)) U
//                                        A = K^T (transposed LDS reads), B = U
//   O^T = scale ((S_0^T Q^T) diag(exp G) + U^T P^T)
//        P = (Q K^T) exp(G_r - G_s) on s <= r, zero above
//
// The products take their operands straight from registers: a C-layout
// result read with the contraction index permuted by perm_row is a B
// operand over its rows, and, transposed, an A operand over its rows.  So
// S_0 (as B of Y and A of S_0^T Q^T), Z, and U (as B of the state update and
// A of U^T P^T) never move between lanes.  K and Q are staged twice over
// where needed: with their dk columns permuted (phi_col_pos) so that an
// A-operand fragment of K or Q is one 16-byte LDS read, and K also in
// natural order for the transposed reads of K^T.  The P tiles are computed
// as K Q^T, whose accumulator layout is the P operand's, split over the
// waves and shared through LDS.
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

namespace la {

enum : int { kXScan = 0, kXReplay = 1, kXMap = 2 };

// Columns per workgroup: a whole 128-column head on four waves; 64 columns
// on two waves when a head dimension is 64 (the map's Phi and R parts then
// split at a part boundary).
template <int DK, int DV> constexpr int xscan_cols() { return (DK == 128 && DV == 128) ? 128 : 64; }

template <int DK, int CW> struct XLds {
    static constexpr int LDP = DK + 8;   // bf16 row pitch, K and Q with permuted dk columns
    static constexpr int LDN = DK + 8;   // bf16 row pitch, K in natural order (transposed reads)
    static constexpr int LDV = CW + 8;   // bf16 row pitch, V
    struct Buf {
        __bf16 kp[kChunk][LDP];
        __bf16 kn[kChunk][LDN];
        __bf16 qp[kChunk][LDP];
        __bf16 v[kChunk][LDV];
        uint4 xf[kXFrags][64];
        float gb[kGateBlock];
    };
    Buf buf[2];
    uint4 pf[4][2][64];   // P fragments [row tile][k-step][lane]
};

// Position of dk column d in the permuted rows: A-operand k-step ks of lane
// group g takes columns perm_row(8 ks + j, g), j < 8, which sit at
// 32 ks + 8 g + j.
__device__ inline int xperm_pos8(int m) {
    // start of the first 4-run of the 8 columns 8m .. 8m + 7 (the second
    // run sits 8 further on)
    return 32 * (m >> 2) + 16 * (m & 1) + 4 * ((m >> 1) & 1);
}

// A-operand fragment of K^T for dk rows [n0, n0 + 16) and k-step ks, the
// chunk rows permuted by perm_row: lane (g, r) takes K[perm_row(8 ks + j, g)][n0 + r],
// two runs of 4 rows (32 ks + 4 g and 32 ks + 16 + 4 g), each one transposed
// LDS read from the natural-order rows.
__device__ inline bf16x8 kt_frag(const __bf16 *kn, int ld, int ks, int n0, int lane) {
    typedef short i16x8 __attribute__((ext_vector_type(8)));
    const int g = lane >> 4, s = lane & 15;
    const auto lo = RowTile<__bf16>::tr4(kn, ld, 32 * ks + 4 * g + (s >> 2), n0, lane);
    const auto hi = RowTile<__bf16>::tr4(kn, ld, 32 * ks + 16 + 4 * g + (s >> 2), n0, lane);
    const i16x8 both = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, both);
}

template <int DK, int DV, int MODE>
__global__ __launch_bounds__((2 * xscan_cols<DK, DV>())) void gdr_xscan_kernel(ScanArgs a) {
    using M = MT<__bf16>;
    using RTl = RowTile<__bf16>;
    typedef __bf16 T;
    constexpr int CW = xscan_cols<DK, DV>();
    constexpr int NWV = CW / 32;                       // waves
    constexpr int NTH = 64 * NWV;                      // threads
    constexpr int RT = DK / 16, FS = DK / 4, KS = DK / 32;
    constexpr int NCOLS = (MODE == kXMap) ? DK + DV : DV;   // column space of the unit
    constexpr int NP = NCOLS / CW;                     // parts per (sequence, head[, segment])
    constexpr bool kOut = MODE != kXMap;
    static_assert(NP * CW == NCOLS && (MODE != kXMap || DK % CW == 0), "column parts");
    using Lds = XLds<DK, CW>;
    constexpr int LDN = Lds::LDN, LDV = Lds::LDV;
    __shared__ Lds sm;

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, c16 = lane & 15;
    const int H = a.n_heads;

    // ---- unit: (sequence, head[, segment], part); the parts of one chain
    // (or segment) share an XCD and its L2
    int pair, sg = 0;
    const int b = blockIdx.x, xcd = b & 7, qb = b >> 3;
    const int part = qb % NP, chain = xcd + 8 * (qb / NP);
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
    const int vcol0 = (MODE == kXMap) ? cb - DK : cb;  // first value column of the part (R / state)

    // ---- state: this wave's two column tiles, all DK rows
    f32x4 S[2][RT];
    if constexpr (MODE == kXMap) {
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    S[c][t][i] = (phi && 16 * t + 4 * g16 + i == cb + 32 * w + 16 * c + c16) ? 1.f : 0.f;
    } else if (MODE == kXReplay && sg > 0) {
        const float *src = a.seg.state + (seg_slot * H + h) * DK * DV;
#pragma unroll
        for (int c = 0; c < 2; ++c) load_state_c<RT>(src, (vcol0 + 32 * w + 16 * c) / 16, S[c]);
    } else {
        const float *src = start_state(a, seq, h, (size_t)DK * DV, part == 0 && w == 0);
#pragma unroll
        for (int c = 0; c < 2; ++c) load_state_tile<DK, DV>(src, (vcol0 + 32 * w) / 16 + c, S[c]);
    }
    float dprod = 1.f;   // product of the chunk decays (the map's D)

    // P fragments above the diagonal that no P tile writes stay zero
    if constexpr (kOut) {
        for (int e = tid; e < 4 * 2 * 64; e += NTH) (&sm.pf[0][0][0])[e] = make_uint4(0, 0, 0, 0);
    }

    // ---- staging: chunk jj's inputs into registers, then into LDS buffer
    constexpr int KP = kChunk * DK / 8;                // 16-byte pieces of K (and of Q)
    constexpr int VP = kChunk * CW / 8;                // pieces of the part's V columns
    constexpr int XP = kXFrags * 64, GP = kGateBlock / 4;
    constexpr int NK = (KP + NTH - 1) / NTH, NV = (VP + NTH - 1) / NTH;
    constexpr int NX = (XP + NTH - 1) / NTH, NG = (GP + NTH - 1) / NTH;
    static_assert(KP % NTH == 0 && VP % NTH == 0, "staging tiling");
    struct Stage {
        uint4 k[NK], q[kOut ? NK : 1], v[NV], x[NX], gbv[NG];
    };
    const T *qin = (const T *)a.q, *kin = (const T *)a.k, *vin = (const T *)a.v;
    const bool has_v = !phi;
    auto load = [&](Stage &st, int jj) {
        int lo, hi;
        chunk_range32(jj, len, a.C, a.cps, &lo, &hi);
        const int n = hi - lo;
        const int64_t t0 = (int64_t)cu0 + lo;
        const int64_t sh = (base + jj) * H + h;
#pragma unroll
        for (int it = 0; it < NK; ++it) {
            const int e = tid + NTH * it, r = e / (DK / 8), c = 8 * (e % (DK / 8));
            const int64_t row = (t0 + min(r, n - 1)) * H + h;
            st.k[it] = *(const uint4 *)(kin + row * DK + c);
            if constexpr (kOut) st.q[it] = *(const uint4 *)(qin + row * DK + c);
            if (r >= n) {
                st.k[it] = make_uint4(0, 0, 0, 0);
                if constexpr (kOut) st.q[it] = make_uint4(0, 0, 0, 0);
            }
        }
#pragma unroll
        for (int it = 0; it < NV; ++it) {
            const int e = tid + NTH * it, r = e / (CW / 8), c = 8 * (e % (CW / 8));
            st.v[it] = make_uint4(0, 0, 0, 0);
            if (has_v && r < n) st.v[it] = *(const uint4 *)(vin + ((t0 + r) * H + h) * DV + vcol0 + c);
        }
        const uint4 *xs = (const uint4 *)a.ws.xf + sh * XP;
#pragma unroll
        for (int it = 0; it < NX; ++it) {
            const int e = tid + NTH * it;
            if (e < XP) st.x[it] = xs[e];
        }
        const uint4 *gs = (const uint4 *)(a.ws.gb + sh * kGateBlock);
#pragma unroll
        for (int it = 0; it < NG; ++it) {
            const int e = tid + NTH * it;
            if (e < GP) st.gbv[it] = gs[e];
        }
    };
    auto store = [&](const Stage &st, int bi) {
        typename Lds::Buf &B = sm.buf[bi];
#pragma unroll
        for (int it = 0; it < NK; ++it) {
            const int e = tid + NTH * it, r = e / (DK / 8), m = e % (DK / 8);
            *(uint4 *)&B.kn[r][8 * m] = st.k[it];
            const int p = xperm_pos8(m);
            *(uint2 *)&B.kp[r][p] = make_uint2(st.k[it].x, st.k[it].y);
            *(uint2 *)&B.kp[r][p + 8] = make_uint2(st.k[it].z, st.k[it].w);
            if constexpr (kOut) {
                *(uint2 *)&B.qp[r][p] = make_uint2(st.q[it].x, st.q[it].y);
                *(uint2 *)&B.qp[r][p + 8] = make_uint2(st.q[it].z, st.q[it].w);
            }
        }
#pragma unroll
        for (int it = 0; it < NV; ++it) {
            const int e = tid + NTH * it, r = e / (CW / 8), c = 8 * (e % (CW / 8));
            *(uint4 *)&B.v[r][c] = st.v[it];
        }
#pragma unroll
        for (int it = 0; it < NX; ++it) {
            const int e = tid + NTH * it;
            if (e < XP) (&B.xf[0][0])[e] = st.x[it];
        }
#pragma unroll
        for (int it = 0; it < NG; ++it) {
            const int e = tid + NTH * it;
            if (e < GP) ((uint4 *)B.gb)[e] = st.gbv[it];
        }
    };

    // ---- checkpoints (single-level scan only)
    CkptDst ck;
    if constexpr (MODE == kXScan) ck.init(a, seq, h, len, (size_t)DK * DV, part == 0 && w == 0);
    uint32_t lane_off[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) lane_off[c] = 4u * (uint32_t)(4 * g16 * DV + vcol0 + 32 * w + 16 * c + c16);

    const float scale = a.scale;
    Stage st;
    load(st, c0);
    store(st, 0);
    __syncthreads();

    for (int jj = c0; jj < c1; ++jj) {
        const int bi = (jj - c0) & 1;
        const typename Lds::Buf &B = sm.buf[bi];
        if (jj + 1 < c1) load(st, jj + 1);
        int lo, hi;
        chunk_range32(jj, len, a.C, a.cps, &lo, &hi);
        const int n = hi - lo;

        // S_0 as B operand (and A operand of S_0^T), dk permuted by perm_row
        T sb[2][FS];
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int f = 0; f < FS; ++f) sb[c][f] = (T)S[c][f >> 2][f & 3];

        // ---- Y = K S_0, O^T = S_0^T Q^T, and this wave's P tiles, by row tile
        f32x4 Y[2][4], O[2][4];
        typename M::frag kf[4][KS];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kf[mt][ks] = M::pack(&B.kp[16 * mt + c16][32 * ks + 8 * g16]);
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                Y[c][mt] = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) Y[c][mt] = M::mma(kf[mt][ks], M::pack(&sb[c][8 * ks]), Y[c][mt]);
            }
            if constexpr (kOut) {
                typename M::frag qf[KS];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) qf[ks] = M::pack(&B.qp[16 * mt + c16][32 * ks + 8 * g16]);
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    O[c][mt] = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) O[c][mt] = M::mma(M::pack(&sb[c][8 * ks]), qf[ks], O[c][mt]);
                }
                // P tiles (mt, nt), nt <= mt: tile index mt (mt + 1) / 2 + nt,
                // dealt to the waves round-robin
#pragma unroll
                for (int nt = 0; nt <= mt; ++nt) {
                    if ((mt * (mt + 1) / 2 + nt) % NWV != w) continue;   // wave-uniform
                    f32x4 p = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) p = M::mma(kf[nt][ks], qf[ks], p);
                    // lane (g, c): P[r = 16 mt + c][s = 16 nt + 4 g + i]
                    const float gr = B.gb[16 * mt + c16] * kLog2e;
                    const float4 gs = *(const float4 *)&B.gb[16 * nt + 4 * g16];
                    const float gsv[4] = {gs.x, gs.y, gs.z, gs.w};
                    T pv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int s = 16 * nt + 4 * g16 + i, r = 16 * mt + c16;
                        pv[i] = (T)(s <= r ? p[i] * __builtin_amdgcn_exp2f(gr - gsv[i] * kLog2e) : 0.f);
                    }
                    *(uint2 *)((char *)&sm.pf[mt][nt >> 1][lane] + 8 * (nt & 1)) = *(const uint2 *)pv;
                }
            }
        }

        // ---- Z = diag(beta) V - diag(d) Y, then U = X Z
        f32x4 U[2][4];
        {
            T zb[2][16];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const float4 d4 = *(const float4 *)&B.gb[kChunk + 16 * mt + 4 * g16];
                const float4 b4 = *(const float4 *)&B.gb[2 * kChunk + 16 * mt + 4 * g16];
                const float dv[4] = {d4.x, d4.y, d4.z, d4.w}, bv[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    float vv[4] = {0.f, 0.f, 0.f, 0.f};
                    if (has_v) {
                        float o4[4];
                        RTl::col4(&B.v[0][0], LDV, mt, 32 * w + 16 * c, lane, o4);
#pragma unroll
                        for (int i = 0; i < 4; ++i) vv[i] = o4[i];
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) zb[c][4 * mt + i] = (T)(bv[i] * vv[i] - dv[i] * Y[c][mt][i]);
                }
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    U[c][mt] = zero4();
#pragma unroll
                    for (int ks = 0; ks <= (mt >> 1); ++ks)
                        U[c][mt] = M::mma(M::pack((const T *)&B.xf[xfrag_slot(mt, ks)][lane]), M::pack(&zb[c][8 * ks]),
                                          U[c][mt]);
                }
        }

        // ---- state update: S = exp(G_63) S + K^T diag(exp(G_63 - G)) U
        T ub[2][16], ub2[2][16];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const float4 e4 = *(const float4 *)&B.gb[3 * kChunk + 16 * mt + 4 * g16];
            const float ev[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    ub[c][4 * mt + i] = (T)U[c][mt][i];
                    ub2[c][4 * mt + i] = (T)(U[c][mt][i] * ev[i]);
                }
        }
        const float eL = __builtin_amdgcn_exp2f(B.gb[kChunk - 1] * kLog2e);
        dprod *= eL;
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            typename M::frag kt[2];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) kt[ks] = kt_frag(&B.kn[0][0], LDN, ks, 16 * t, lane);
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                f32x4 acc = S[c][t] * eL;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) acc = M::mma(kt[ks], M::pack(&ub2[c][8 * ks]), acc);
                S[c][t] = acc;
            }
        }
        if constexpr (MODE == kXScan) {
            // checkpoint when the chunk ends on a multiple of C (positions are
            // local and start on a multiple of C)
            if (hi % a.C == 0) {
                if (float *d = ck.next(ck.load_id(hi / a.C - 1))) {
#pragma unroll
                    for (int c = 0; c < 2; ++c) store_state_tiles<RT, DV>(d, S[c], lane_off[c]);
                }
            }
        }

        if constexpr (kOut) {
            lds_barrier();   // every wave's P tiles are in LDS
            // ---- O^T = scale ((S_0^T Q^T) diag(exp G) + U^T P^T), stored 4 columns per lane
            T *obase = (T *)a.o + (((int64_t)cu0 + lo) * H + h) * DV;
            const auto ro = make_rsrc(obase, head_rows_bytes<T>(n, H, DV));
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const float eg = __builtin_amdgcn_exp2f(B.gb[16 * mt + c16] * kLog2e);
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    f32x4 acc = O[c][mt] * eg;
#pragma unroll
                    for (int ks = 0; ks <= (mt >> 1); ++ks)
                        acc = M::mma(M::pack(&ub[c][8 * ks]), M::pack((const T *)&sm.pf[mt][ks][lane]), acc);
                    T out[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) out[i] = (T)(acc[i] * scale);
                    const uint32_t voff = ((uint32_t)(16 * mt + c16) * (uint32_t)(H * DV) +
                                           (uint32_t)(vcol0 + 32 * w + 16 * c + 4 * g16)) * (uint32_t)sizeof(T);
                    buf_store8(*(const uint2 *)out, ro, voff, 0u);
                }
            }
        }
        // chunk jj + 1's inputs into the other buffer; every wave has
        // finished reading it (chunk jj - 1) before the last barrier
        if (jj + 1 < c1) store(st, bi ^ 1);
        lds_barrier();
    }

    // ---- epilogue
    if constexpr (MODE == kXScan) {
        if (a.final_state) {
#pragma unroll
            for (int c = 0; c < 2; ++c)
                store_state_tiles<RT, DV>(a.final_state + (size_t)pair * DK * DV, S[c], lane_off[c]);
        }
    }
    if constexpr (MODE == kXMap) {
        const int64_t ssh = seg_slot * H + h;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int col = cb + 32 * w + 16 * c + c16;
            if (phi) {
                T *dst = (T *)a.seg.phi + ssh * DK * DK + phi_col_pos(col);
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int r = 16 * t + 4 * g16 + e;
                        dst[(size_t)r * DK] = (T)(S[c][t][e] - (r == col ? dprod : 0.f));
                    }
            } else {
                float4 *dst = (float4 *)(a.seg.r + ssh * DK * DV);
                const int tile = (col - DK) / 16;
#pragma unroll
                for (int t = 0; t < RT; ++t)
                    dst[(tile * RT + t) * 64 + lane] = make_float4(S[c][t][0], S[c][t][1], S[c][t][2], S[c][t][3]);
            }
        }
        if (part == 0 && w == 0 && lane == 0) a.seg.d[ssh] = dprod;
    }
}

}  // namespace la

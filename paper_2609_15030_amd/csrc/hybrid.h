// Joint restore of a hybrid cache at one boundary B: for every sequence, the
// attention KV blocks of its prefix [0, B) and the recurrent state pages of
// its checkpoint at B, in one launch.  A hybrid model's reload moves both
// kinds of entries (section 2.1; Table 5), and they are usable together
// only when the attention prefix and the checkpoint describe the same
// prefix (sections 1 and 6).
//
// Workgroup (x, y, z) serves sequence y.  x < nb_max: its KV block x, if x <
// B_y / block_tokens (cache[dst] = pool[src]); nb_max <= x < nb_max + H: its
// state page for head x - nb_max (states = pool page; id -1: zero state).
// z selects one part of kHybridPartVec 16-byte vectors of the item, so a
// restore of a few hundred 100-KB blocks still spreads over about a
// thousand workgroups, each with all its loads in flight at once
// (non-temporal loads, then ordinary stores).  KV blocks are opaque bytes.
// Ids out of range skip the item and are counted once (by part 0).
#pragma once
#include "paged.h"

namespace la {

constexpr int kHybridPartVec = 2 * kPageThreads;   // 32 KiB per workgroup

// Copies vectors [lo, hi) (at most kHybridPartVec): every load first.
__device__ inline void copy_part(const f32x4 *__restrict__ src, f32x4 *__restrict__ dst, int64_t lo, int64_t hi) {
    const int64_t v0 = lo + threadIdx.x, v1 = v0 + kPageThreads;
    f32x4 x0 = zero4(), x1 = zero4();
    if (v0 < hi) x0 = __builtin_nontemporal_load(src + v0);
    if (v1 < hi) x1 = __builtin_nontemporal_load(src + v1);
    if (v0 < hi) dst[v0] = x0;
    if (v1 < hi) dst[v1] = x1;
}

struct HybridArgs {
    const f32x4 *kv_pool;        // [n_pool_blocks][kv_vec]
    f32x4 *cache;                // [n_cache_blocks][kv_vec]
    const int32_t *src_ids, *dst_ids;   // [n_seqs][max_blocks]
    const int64_t *boundary;     // [n_seqs]
    const f32x4 *state_pool;     // [n_state_pages][page_vec]
    const int32_t *state_ids;    // [n_seqs * H]
    f32x4 *states;               // [n_seqs * H][page_vec]
    int32_t *err;
    int64_t kv_vec, n_pool_blocks, n_cache_blocks, max_blocks, block_tokens;
    int64_t page_vec, n_state_pages;
    int32_t n_heads, nb_max;
};

__global__ __launch_bounds__(kPageThreads) void hybrid_restore_kernel(HybridArgs a) {
    const int64_t seq = blockIdx.y;
    const int x = blockIdx.x;
    const int64_t lo = (int64_t)blockIdx.z * kHybridPartVec;
    const bool counter = blockIdx.z == 0 && threadIdx.x == 0 && a.err;
    if (x < a.nb_max) {
        if (x >= a.boundary[seq] / a.block_tokens || lo >= a.kv_vec) return;
        const int32_t s = a.src_ids[seq * a.max_blocks + x], d = a.dst_ids[seq * a.max_blocks + x];
        if (s == -1 || d == -1) return;
        if (s < 0 || s >= a.n_pool_blocks || d < 0 || d >= a.n_cache_blocks) {
            if (counter) atomicAdd(a.err, 1);
            return;
        }
        copy_part(a.kv_pool + (int64_t)s * a.kv_vec, a.cache + (int64_t)d * a.kv_vec, lo,
                  min(lo + kHybridPartVec, a.kv_vec));
        return;
    }
    if (lo >= a.page_vec) return;
    const int64_t hi = min(lo + kHybridPartVec, a.page_vec);
    const int64_t item = seq * a.n_heads + (x - a.nb_max);
    const int32_t pid = a.state_ids[item];
    f32x4 *dst = a.states + item * a.page_vec;
    if (pid == -1) {
        for (int64_t v = lo + threadIdx.x; v < hi; v += kPageThreads) dst[v] = zero4();
        return;
    }
    if (pid < 0 || pid >= a.n_state_pages) {
        if (counter) atomicAdd(a.err, 1);
        return;
    }
    copy_part(a.state_pool + (int64_t)pid * a.page_vec, dst, lo, hi);
}

}  // namespace la

// Bookkeeping between rounds (Appendix C stages I, II and IV):
//
// * commit_kv_kernel: the root (the last committed token) and the accepted
//   draft tokens become part of the committed prefix, so their tree K/V rows
//   are appended, in path order, to each sequence's cache slot, and the
//   slot's length advances on the device (no host round trip).
// * select_slots_kernel: in quadratic self-speculation the next round's
//   drafter rows are the mask slots hanging off the last accepted node; this
//   writes their row indices into the slot-logit matrix, for presto_topk_rows
//   to read in place (no copy of V-wide rows).
// * flatten_slots_kernel: the next forward's composite input puts a block of
//   mask slots after every draft node; this writes the positions and the
//   attention mask of that layout (node rows see their root path, slot rows
//   see their node's root path and their whole block).
#include "common.hpp"

namespace presto {

constexpr int kCommitThreads = 512;

// One workgroup per sequence: validate, copy (1 + accept_len) rows of K and
// of V, then advance the length.  row16 = bytes of one [hkv, head_dim] row / 16.
__global__ __launch_bounds__(kCommitThreads) void commit_kv_kernel(
    const uint4* __restrict__ kt, const uint4* __restrict__ vt, const int32_t* __restrict__ path,
    const int32_t* __restrict__ accept_len, uint4* __restrict__ kc, uint4* __restrict__ vc,
    int64_t cache_rows, int32_t* __restrict__ ctx, const int32_t* __restrict__ ctx_cap,
    int32_t n_max, int32_t depth, int32_t row16, int32_t* __restrict__ flags) {
    const int b = blockIdx.x, tid = threadIdx.x;
    const int32_t start = ctx[2 * b], len = ctx[2 * b + 1], cap = ctx_cap[b];
    const int32_t al = accept_len[b];
    const int32_t* pb = path + (int64_t)b * (depth + 1);
    const int m = al + 1;
    bool bad = al < 0 || al > depth || start < 0 || len < 0 || cap < 0 ||
               (int64_t)start + cap > cache_rows || (int64_t)len + m > cap;
    // every path entry is checked, whatever the depth (a path may be longer
    // than the workgroup)
    for (int i = tid; !bad && i < m; i += kCommitThreads) {
        const int32_t node = pb[i];
        bad = node < 0 || node >= n_max || (i == 0 && node != 0);
    }
    if (__syncthreads_or(bad)) {
        if (tid == 0) raise_flag(flags, PRESTO_FLAG_KV_COMMIT);
        return;
    }
    const int64_t dst0 = ((int64_t)start + len) * row16;
    const int total = m * row16;
    for (int i = tid; i < total; i += kCommitThreads) {
        const int r = i / row16, c = i - r * row16;
        const int64_t src = ((int64_t)b * n_max + pb[r]) * row16 + c;
        const int64_t dst = dst0 + (int64_t)r * row16 + c;
        const uint4 kv = kt[src], vv = vt[src];
        kc[dst] = kv;
        vc[dst] = vv;
    }
    __syncthreads();  // every lane has read the old length
    if (tid == 0) ctx[2 * b + 1] = len + m;
}

// row_index[b, d] = row of slot (first_slot + d) of the last accepted node of
// sequence b in the slot-logit matrix [batch, n_max, slots, V].
__global__ void select_slots_kernel(int32_t batch, int32_t n_max, int32_t depth, int32_t slots,
                                    int32_t first_slot, const int32_t* __restrict__ path,
                                    const int32_t* __restrict__ accept_len,
                                    int64_t* __restrict__ row_index, int32_t* __restrict__ flags) {
    const int rows = slots - first_slot;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)batch * rows) return;
    const int b = (int)(i / rows), d = (int)(i % rows);
    const int32_t al = accept_len[b];
    int32_t last = (al >= 0 && al <= depth) ? path[(int64_t)b * (depth + 1) + al] : -1;
    if (last < 0 || last >= n_max) {
        if (d == 0) raise_flag(flags, PRESTO_FLAG_KV_COMMIT);
        last = 0;  // fall back to the root's block
    }
    row_index[i] = ((int64_t)b * n_max + last) * slots + first_slot + d;
}

// One lane per (composite row, mask word).  Composite row r = n * (1 + S) + j:
// node n (j = 0) or its slot j (1 .. S).  Column c = m * (1 + S) + jj.  The
// node columns of a word (jj = 0) are consecutive nodes m0 .. m1, so their
// bits are one field of node n's ancestor row, spread out (1 + S) apart; the
// slot columns a slot row sees are one range, its own block.
__global__ void flatten_slots_kernel(int32_t batch, int32_t n_max, int32_t S,
                                     const int32_t* __restrict__ depth,
                                     const uint64_t* __restrict__ anc,
                                     const int32_t* __restrict__ n_nodes,
                                     const int32_t* __restrict__ root_pos,
                                     int32_t* __restrict__ pos_out, uint64_t* __restrict__ anc_out,
                                     int32_t* __restrict__ n_rows) {
    const int blk = 1 + S;
    const int R = n_max * blk;
    const int W = (n_max + 63) / 64, WO = (R + 63) / 64;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)batch * R * WO) return;
    const int w = (int)(i % WO);
    const int r = (int)((i / WO) % R);
    const int b = (int)(i / ((int64_t)WO * R));
    const int n = r / blk, j = r - n * blk;
    int nn = n_nodes[b];
    nn = nn < 0 ? 0 : (nn > n_max ? n_max : nn);
    const bool live = n < nn;
    if (w == 0) {
        pos_out[(int64_t)b * R + r] = live ? root_pos[b] + depth[(int64_t)b * n_max + n] + j : -1;
        if (r == 0) n_rows[b] = nn * blk;
    }
    uint64_t bits = 0;
    if (live) {
        const int c0 = 64 * w, c1 = min(c0 + 64, R);  // columns [c0, c1)
        // node columns m * blk in [c0, c1) with m < nn: at most 32 (blk >= 2)
        const int m0 = (c0 + blk - 1) / blk;
        const int m1 = min((c1 - 1) / blk, nn - 1);
        if (m0 <= m1) {
            const uint64_t* arow = anc + ((int64_t)b * n_max + n) * W;
            const int wa = m0 >> 6, sh = m0 & 63;
            uint64_t f = arow[wa] >> sh;
            if (sh != 0 && wa + 1 < W) f |= arow[wa + 1] << (64 - sh);
            for (int q = 0; q <= m1 - m0; ++q) bits |= ((f >> q) & 1ull) << ((m0 + q) * blk - c0);
        }
        // a slot row sees its whole block: columns n * blk + 1 .. n * blk + S
        if (j > 0) {
            const int s0 = max(n * blk + 1, c0), s1 = min(n * blk + S + 1, c1);  // [s0, s1)
            if (s0 < s1) {
                const int len = s1 - s0;
                bits |= (len == 64 ? ~0ull : (1ull << len) - 1ull) << (s0 - c0);
            }
        }
    }
    anc_out[((int64_t)b * R + r) * WO + w] = bits;
}

}  // namespace presto

namespace presto_host {

using namespace presto;

presto_status launch_commit_kv(const presto_commit_desc* d, const void* k_tree, const void* v_tree,
                               const int32_t* path, const int32_t* accept_len, void* k_cache,
                               void* v_cache, int64_t cache_rows, int32_t* ctx,
                               const int32_t* ctx_cap, int32_t* flags, hipStream_t stream) {
    const int esz = d->dt == PRESTO_DT_BF16 ? 2 : 4;
    const int32_t row16 = d->hkv * d->head_dim * esz / 16;
    commit_kv_kernel<<<d->batch, kCommitThreads, 0, stream>>>(
        static_cast<const uint4*>(k_tree), static_cast<const uint4*>(v_tree), path, accept_len,
        static_cast<uint4*>(k_cache), static_cast<uint4*>(v_cache), cache_rows, ctx, ctx_cap,
        d->n_max, d->depth, row16, flags);
    return check_launch("commit_kv_kernel");
}

presto_status launch_select_slots(int32_t batch, int32_t n_max, int32_t depth, int32_t slots,
                                  int32_t first_slot, const int32_t* path,
                                  const int32_t* accept_len, int64_t* row_index, int32_t* flags,
                                  hipStream_t stream) {
    const int64_t total = (int64_t)batch * (slots - first_slot);
    select_slots_kernel<<<(unsigned)((total + 255) / 256), 256, 0, stream>>>(
        batch, n_max, depth, slots, first_slot, path, accept_len, row_index, flags);
    return check_launch("select_slots_kernel");
}

presto_status launch_flatten_slots(int32_t batch, int32_t n_max, int32_t slots,
                                   const int32_t* depth, const uint64_t* anc,
                                   const int32_t* n_nodes, const int32_t* root_pos,
                                   int32_t* pos_out, uint64_t* anc_out, int32_t* n_rows,
                                   hipStream_t stream) {
    const int64_t R = (int64_t)n_max * (1 + slots);
    const int64_t total = (int64_t)batch * R * ((R + 63) / 64);
    flatten_slots_kernel<<<(unsigned)((total + 255) / 256), 256, 0, stream>>>(
        batch, n_max, slots, depth, anc, n_nodes, root_pos, pos_out, anc_out, n_rows);
    return check_launch("flatten_slots_kernel");
}

}  // namespace presto_host

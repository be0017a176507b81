// NEXT-4 -- incremental re-validation of selector rows after node-label
// changes (paper, Abstract: the validator is meant for continuous
// cross-layer compliance checking).  Instead of rebuilding every row's
// bitset, only the listed nodes' bits are re-evaluated.  Also the
// membership probes of verdict-only runs (one (row, node) query a thread).
//
// Design (gfx950):
//   1. validate : NODE over the list.
//   2. prep     : one workgroup sorts the in-range listed nodes (bitonic, in
//                 LDS), drops repeats, and gathers their label rows into a
//                 compact block.  A node's new bit depends only on its new
//                 labels, so a repeated node changes nothing more.
//   3. rows     : one thread per row, which also raises the rows' PRED /
//                 OFFSETS flags (as pc_eval_selectors); the workgroup stages
//                 the label rows of 64 nodes at a time in LDS.  Each
//                 predicate of the row is loaded once per batch and tested
//                 on every node of it into a 64-bit node mask; the masks are
//                 AND-ed, and each bitset word the batch touches is updated
//                 (plainly, and only when a listed bit changes, when there is
//                 one batch; else with one atomic clear that returns the old
//                 word and one atomic set), the popcount moving by the
//                 words' change.
#include <climits>
#include <cstdlib>

#include "pc_internal.h"

namespace {

constexpr int kUpdMax = PC_UPDATE_MAX_NODES;  // listed nodes per call
constexpr int kPrepThreads = 1024;
constexpr int kRowThreads = 256;             // one row per thread

__device__ __forceinline__ bool upd_pred_valid(const pc_pred &q, int32_t L)
{
    return static_cast<int32_t>(q.label) < L && q.op <= PC_OP_EXISTS && q.rsv0 == 0 && q.rsv1 == 0 &&
           (q.op == PC_OP_EXISTS || (q.vals[3] >> 63) == 0);
}

__global__ __launch_bounds__(256) void k_upd_validate(const int32_t *__restrict__ pred_off,
                                                      const pc_pred *__restrict__ preds, int64_t n_preds, int32_t I,
                                                      int32_t L, const int32_t *__restrict__ nodes, int32_t M, int32_t N,
                                                      uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    const int64_t tot = I > M ? I : M;
    for (int64_t x = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; x < tot;
         x += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (x < I) {
            const int64_t b = pred_off[x], e = pred_off[x + 1];
            if (!pc_range_ok(b, e, n_preds)) {
                errs |= PC_DERR_OFFSETS;
            } else {
                for (int64_t p = b; p < e; ++p)
                    if (!upd_pred_valid(preds[p], L)) {
                        errs |= PC_DERR_PRED;
                        break;
                    }
            }
        }
        if (x < M && (nodes[x] < 0 || nodes[x] >= N)) errs |= PC_DERR_NODE;
    }
    if (errs) atomicOr(d_err, errs);
}

// Sorted distinct in-range nodes -> uniq[0..*d_mu), their label rows ->
// ulab[k * L ...].
// n2: a power of two >= M (at most kUpdMax); only key[0..n2) is sorted.
__global__ __launch_bounds__(kPrepThreads) void k_upd_prep(const int32_t *__restrict__ nodes, int32_t M, int32_t N,
                                                           const uint8_t *__restrict__ labels, int32_t L,
                                                           int32_t *__restrict__ uniq, uint8_t *__restrict__ ulab,
                                                           int32_t *__restrict__ d_mu, int32_t n2)
{
    __shared__ int32_t key[kUpdMax];
    __shared__ int32_t comp[kUpdMax];
    __shared__ int32_t wsum[kPrepThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    for (int i = tid; i < kUpdMax; i += kPrepThreads) {
        const int32_t n = i < M ? nodes[i] : -1;
        key[i] = (n >= 0 && n < N) ? n : INT32_MAX;
    }
    __syncthreads();
    // bitonic sort of key[0..n2), ascending (the rest holds INT32_MAX)
    for (int k = 2; k <= n2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < n2; i += kPrepThreads) {
                const int l = i ^ j;
                if (l > i) {
                    const int32_t a = key[i], b = key[l];
                    const bool up = (i & k) == 0;
                    if ((a > b) == up) {
                        key[i] = b;
                        key[l] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    // keep the first of each run: positions by an exclusive scan, 4 entries per thread
    constexpr int kPer = kUpdMax / kPrepThreads;
    int flag[kPer], cnt = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int i = tid * kPer + k;
        flag[k] = key[i] != INT32_MAX && (i == 0 || key[i - 1] != key[i]);
        cnt += flag[k];
    }
    int x = cnt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wsum[wid] = x;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wid; ++w) base += wsum[w];
    int pos = base + x - cnt;
#pragma unroll
    for (int k = 0; k < kPer; ++k)
        if (flag[k]) {
            comp[pos] = key[tid * kPer + k];
            uniq[pos] = key[tid * kPer + k];
            ++pos;
        }
    if (tid == kPrepThreads - 1) *d_mu = pos;
    __syncthreads();
    int mu = 0;
    for (int w = 0; w < kPrepThreads / 64; ++w) mu += wsum[w];
    for (int64_t i = tid; i < static_cast<int64_t>(mu) * L; i += kPrepThreads) {
        const int64_t k = i / L, l = i % L;
        ulab[i] = labels[static_cast<int64_t>(comp[k]) * L + l];
    }
}

// One thread per row (see the file header).  The row's offset pair and
// predicates are validated first (PRED / OFFSETS as pc_eval_selectors);
// then, per batch of up to 64 sorted nodes staged in LDS, each predicate is
// loaded once and tested on every node of the batch into a 64-bit node
// mask, the masks are AND-ed, and the row's bitset words are updated word
// by word (the nodes are sorted, so a word's nodes are consecutive).
__global__ __launch_bounds__(kRowThreads) void k_upd_rows(const int32_t *__restrict__ pred_off,
                                                          const pc_pred *__restrict__ preds, int64_t n_preds,
                                                          int32_t I, int32_t L, const int32_t *__restrict__ uniq,
                                                          const uint8_t *__restrict__ ulab,
                                                          const int32_t *__restrict__ d_mu, int32_t W,
                                                          uint64_t *__restrict__ feasible,
                                                          uint32_t *__restrict__ popcnt, uint32_t *__restrict__ d_err)
{
    extern __shared__ uint8_t lab_lds[];  // up to 64 nodes x L bytes, then their ids
    const int tid = threadIdx.x;
    const int32_t r = blockIdx.x * kRowThreads + tid;
    const int32_t mu = *d_mu;
    int32_t *ids = reinterpret_cast<int32_t *>(lab_lds + ((static_cast<int64_t>(64) * L + 3) & ~int64_t(3)));
    const bool live = r < I;
    int64_t b = 0, e = 0;
    bool row_ok = false;
    uint32_t errs = 0;
    if (live) {
        b = pred_off[r];
        e = pred_off[r + 1];
        row_ok = pc_range_ok(b, e, n_preds);
        if (!row_ok) errs |= PC_DERR_OFFSETS;
        if (mu == 0)  // no batch: the predicates are only validated
            for (int64_t p = b; row_ok && p < e; ++p)
                if (!upd_pred_valid(preds[p], L)) {
                    errs |= PC_DERR_PRED;
                    row_ok = false;
                }
    }
    uint32_t delta = 0;
    for (int32_t k0 = 0; k0 < mu; k0 += 64) {
        const int32_t nb = min(64, mu - k0);
        __syncthreads();  // the previous batch is no longer read
        for (int32_t i = tid; i < nb * L; i += kRowThreads) lab_lds[i] = ulab[static_cast<int64_t>(k0) * L + i];
        if (tid < nb) ids[tid] = uniq[k0 + tid];
        __syncthreads();
        if (!live) continue;
        // bit m of `hold`: node m of the batch satisfies the row.  The first
        // batch also validates every predicate (a malformed one admits no
        // node and raises PRED), so it reads them all.
        uint64_t hold = nb == 64 ? ~0ull : ((1ull << nb) - 1);
        if (!row_ok) hold = 0;
        const bool first = k0 == 0;
        for (int64_t p = b; row_ok && (hold || first) && p < e; ++p) {
            const pc_pred q = preds[p];
            if (first && !upd_pred_valid(q, L)) {
                errs |= PC_DERR_PRED;
                row_ok = false;
                hold = 0;
                break;
            }
            if (!hold) continue;
            uint64_t m = 0;
            for (int32_t j = 0; j < nb; ++j) {
                const uint32_t x = lab_lds[j * L + q.label];
                const bool present = x != PC_LABEL_ABSENT;
                const uint32_t w = x >> 6;
                const uint64_t vw = w == 0 ? q.vals[0] : w == 1 ? q.vals[1] : w == 2 ? q.vals[2] : q.vals[3];
                const bool in_set = present && ((vw >> (x & 63)) & 1);
                const bool sat = q.op == PC_OP_IN ? in_set : q.op == PC_OP_NOTIN ? !in_set : present;
                m |= static_cast<uint64_t>(sat) << j;
            }
            hold &= m;
        }
        // word by word: the batch's nodes in one word are consecutive
        int32_t j = 0;
        while (j < nb) {
            const int32_t w = ids[j] >> 6;
            uint64_t set = 0, mask = 0;
            for (; j < nb && (ids[j] >> 6) == w; ++j) {
                const uint64_t bit = 1ull << (ids[j] & 63);
                mask |= bit;
                if ((hold >> j) & 1) set |= bit;
            }
            uint64_t *dst = feasible + static_cast<int64_t>(r) * W + w;
            uint64_t old;
            if (mu <= 64) {
                // one batch: every word is touched once, plainly, and written
                // only when one of its listed bits changes
                old = *dst;
                if ((old & mask) != set) *dst = (old & ~mask) | set;
            } else {
                // a word can straddle two batches: the update goes through L2
                // atomics (clear, returning the old word, then set)
                unsigned long long *adst = reinterpret_cast<unsigned long long *>(dst);
                old = atomicAnd(adst, ~(mask & ~set));
                if (set) atomicOr(adst, set);
            }
            const uint64_t nw = (old & ~mask) | set;
            delta += static_cast<uint32_t>(__popcll(nw)) - static_cast<uint32_t>(__popcll(old));
        }
    }
    if (live && delta) popcnt[r] += delta;
    if (errs) atomicOr(d_err, errs);
}

// Membership probes: one thread per (row, node) query, the row's
// predicates evaluated on the node's labels.
__global__ __launch_bounds__(256) void k_probe(const uint8_t *__restrict__ labels, int32_t N, int32_t L,
                                               const int32_t *__restrict__ pred_off, const pc_pred *__restrict__ preds,
                                               int64_t n_preds, int32_t I, const int32_t *__restrict__ probe_row,
                                               const int32_t *__restrict__ probe_node, int32_t P,
                                               uint8_t *__restrict__ bit, uint32_t *__restrict__ d_err)
{
    const int32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= P) return;
    const int32_t r = probe_row[k], n = probe_node[k];
    if (r < 0 || r >= I || n < 0 || n >= N) {
        bit[k] = 0;
        atomicOr(d_err, PC_DERR_NODE);
        return;
    }
    const int64_t b = pred_off[r], e = pred_off[r + 1];
    bool ok = pc_range_ok(b, e, n_preds);
    const uint8_t *lab = labels + static_cast<int64_t>(n) * L;
    for (int64_t p = b; ok && p < e; ++p) {
        const pc_pred q = preds[p];
        if (!upd_pred_valid(q, L)) {
            ok = false;
            break;
        }
        const uint32_t x = lab[q.label];
        const bool present = x != PC_LABEL_ABSENT;
        const uint32_t w = x >> 6;
        const uint64_t vw = w == 0 ? q.vals[0] : w == 1 ? q.vals[1] : w == 2 ? q.vals[2] : q.vals[3];
        const bool in_set = present && ((vw >> (x & 63)) & 1);
        ok = q.op == PC_OP_IN ? in_set : q.op == PC_OP_NOTIN ? !in_set : present;
    }
    bit[k] = ok ? 1 : 0;
}

}  // namespace

int run_probes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
               const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *probe_row,
               const int32_t *probe_node, int32_t P, uint8_t *bit, hipStream_t stream)
{
    if (I > 0) {
        // the rows' flags, as for pc_eval_selectors (no listed nodes)
        const unsigned g = static_cast<unsigned>(std::min<int64_t>((I + 255) / 256, 8192));
        PC_TIMED(ctx, "k_upd_validate", stream,
                 hipLaunchKernelGGL(k_upd_validate, dim3(g), dim3(256), 0, stream, pred_off, preds, n_preds, I, L,
                                    nullptr, 0, N, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (P == 0) return PC_OK;
    PC_TIMED(ctx, "k_probe", stream,
             hipLaunchKernelGGL(k_probe, dim3(static_cast<unsigned>((P + 255) / 256)), dim3(256), 0, stream, labels,
                                N, L, pred_off, preds, n_preds, I, probe_row, probe_node, P, bit, ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

int run_update_nodes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                     const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *nodes, int32_t M,
                     uint64_t *feasible, uint32_t *popcnt, hipStream_t stream)
{
    int32_t *uniq, *d_mu;
    uint8_t *ulab;
    auto carve = [&](Carver &cv) {
        uniq = cv.take<int32_t>(kUpdMax);
        d_mu = cv.take<int32_t>(1);
        ulab = cv.take<uint8_t>(static_cast<size_t>(kUpdMax) * (L > 0 ? L : 1));
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);
    if (M > 0) {
        // NODE over the list (the rows' flags are raised by k_upd_rows)
        const unsigned g = static_cast<unsigned>(std::min<int64_t>((M + 255) / 256, 8192));
        PC_TIMED(ctx, "k_upd_validate", stream,
                 hipLaunchKernelGGL(k_upd_validate, dim3(g), dim3(256), 0, stream, pred_off, preds, n_preds, 0, L,
                                    nodes, M, N, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (I == 0) return PC_OK;
    // Above W / 32 listed nodes the scattered word updates cost about as much
    // as rewriting every row: evaluate the rows in full instead (same result).
    // PC_UPDATE_FULL_ABOVE overrides the threshold.
    const int32_t W = (N + 63) / 64;
    int64_t full_above = W / 32;
    if (const char *env = getenv("PC_UPDATE_FULL_ABOVE")) full_above = atoll(env);
    if (M > full_above && W > 0)
        return run_selectors(ctx, labels, N, L, pred_off, preds, n_preds, I, feasible, popcnt, stream);
    if (M > 0 && N > 0) {
        int32_t n2 = 2;
        while (n2 < M) n2 <<= 1;
        PC_TIMED(ctx, "k_upd_prep", stream,
                 hipLaunchKernelGGL(k_upd_prep, dim3(1), dim3(kPrepThreads), 0, stream, nodes, M, N, labels, L, uniq,
                                    ulab, d_mu, n2));
    } else {
        launch_fill_u32(reinterpret_cast<uint32_t *>(d_mu), 1, 0, stream);
    }
    PC_LAUNCH_CHECK(ctx);
    const size_t lds = ((static_cast<size_t>(64) * L + 3) & ~size_t(3)) + 64 * sizeof(int32_t);
    PC_HIP(ctx, hipFuncSetAttribute(reinterpret_cast<const void *>(k_upd_rows),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    const unsigned g = static_cast<unsigned>((I + kRowThreads - 1) / kRowThreads);
    PC_TIMED(ctx, "k_upd_rows", stream,
             hipLaunchKernelGGL(k_upd_rows, dim3(g), dim3(kRowThreads), lds, stream, pred_off, preds, n_preds, I, L,
                                uniq, ulab, d_mu, W, feasible, popcnt, ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

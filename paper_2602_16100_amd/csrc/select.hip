// A1 -- placement constraints: node-selector evaluation for every selector
// row x node, emitting a feasible-node bitset and a popcount per row.
//
// The operators are Kubernetes node-affinity's (In / NotIn / Exists over a
// label), which is how the paper compiles a placement constraint such as
// "region=EU is among the labels of the node the pod is placed on" (Formal
// Model and Satisfaction, example; Service Placement Module).
//
// Design (gfx950):
//   1. presence  : which values of each label occur at all (LDS-local OR,
//                  one global OR per workgroup).
//   2. label scan: plane numbering -- one plane per present (label, value).
//   3. planes    : planes[p][w] = 64-bit set of nodes 64w..64w+63 carrying
//                  the plane's (label, value); built with one ballot per
//                  present value per 64-node column.
//   4. compile   : one thread per row turns its predicates into a clause
//                  program over plane ids (In S = OR of S's planes or NOT OR
//                  of the rest, whichever is shorter; NotIn the reverse;
//                  Exists = NOT the absent-value plane) and validates it.
//   5. eval      : one row per wavefront (its program read with scalar
//                  loads), lanes over 64 columns of 64 nodes, plane words
//                  fetched kBatch at a time so the loads overlap.  XCD-aware
//                  block -> (column tile, row chunk) mapping keeps each XCD's
//                  planes in its own L2.
#include "pc_internal.h"

namespace {

constexpr int kEvalThreads = 256;     // 4 waves, one row at a time each
constexpr int kPresenceNodes = 4096;  // nodes per presence workgroup

__device__ __forceinline__ uint64_t uniform_u64(uint64_t x)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x >> 32));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__global__ __launch_bounds__(256) void k_sel_presence(const uint8_t *__restrict__ labels, int32_t N, int32_t L,
                                                      int64_t chunk, uint32_t *__restrict__ present32)
{
    __shared__ uint32_t tab[64 * 8];
    const int tid = threadIdx.x;
    for (int i = tid; i < 512; i += 256) tab[i] = 0;
    __syncthreads();
    const int lt = tid & 63, sub = tid >> 6;
    const int32_t l = blockIdx.x * 64 + lt;
    const int64_t n0 = static_cast<int64_t>(blockIdx.y) * chunk;
    const int64_t n1 = min(static_cast<int64_t>(N), n0 + chunk);
    if (l < L) {
        for (int64_t n = n0 + sub; n < n1; n += 4) {
            const uint32_t x = labels[n * L + l];
            atomicOr(&tab[lt * 8 + (x >> 5)], 1u << (x & 31));
        }
    }
    __syncthreads();
    for (int i = tid; i < 512; i += 256) {
        const int32_t ll = blockIdx.x * 64 + (i >> 3);
        if (ll < L && tab[i]) atomicOr(&present32[static_cast<int64_t>(ll) * 8 + (i & 7)], tab[i]);
    }
}

// Exclusive scan of per-label plane counts -> wbase[l][k] = id of the first
// plane of label l whose value lies in 64-value word k.
__global__ __launch_bounds__(1024) void k_sel_label_scan(const uint64_t *__restrict__ present, int32_t L,
                                                         uint32_t *__restrict__ wbase)
{
    __shared__ uint32_t wsum[16];
    __shared__ uint32_t carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int32_t base = 0; base < L; base += 1024) {
        const int32_t l = base + tid;
        uint32_t c[4] = {0, 0, 0, 0};
        if (l < L)
            for (int k = 0; k < 4; ++k) c[k] = __popcll(present[static_cast<int64_t>(l) * 4 + k]);
        const uint32_t v = c[0] + c[1] + c[2] + c[3];
        uint32_t x = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (lane == 63) wsum[wid] = x;
        __syncthreads();
        if (wid == 0) {
            uint32_t w = lane < 16 ? wsum[lane] : 0;
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                uint32_t y = __shfl_up(w, off, 64);
                if (lane >= off) w += y;
            }
            if (lane < 16) wsum[lane] = w;
        }
        __syncthreads();
        const uint32_t carry = carry_s;
        uint32_t excl = carry + (wid ? wsum[wid - 1] : 0) + x - v;
        if (l < L) {
            for (int k = 0; k < 4; ++k) {
                wbase[static_cast<int64_t>(l) * 4 + k] = excl;
                excl += c[k];
            }
        }
        __syncthreads();
        if (tid == 0) carry_s = carry + wsum[15];
        __syncthreads();
    }
}

// One wavefront per (64-node column w, label l): a ballot per present value.
__global__ __launch_bounds__(256) void k_sel_planes(const uint8_t *__restrict__ labels, int32_t N, int32_t L,
                                                    const uint64_t *__restrict__ present,
                                                    const uint32_t *__restrict__ wbase, uint64_t *__restrict__ planes,
                                                    int32_t W)
{
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t w = blockIdx.x;
    const int32_t l = blockIdx.y * 4 + wave;
    if (l >= L) return;
    const int64_t n = static_cast<int64_t>(w) * 64 + lane;
    const uint32_t x = n < N ? labels[n * L + l] : 0x100u;  // 0x100 equals no value
    for (int k = 0; k < 4; ++k) {
        uint64_t m = uniform_u64(present[static_cast<int64_t>(l) * 4 + k]);
        uint32_t pid = __builtin_amdgcn_readfirstlane(wbase[static_cast<int64_t>(l) * 4 + k]);
        while (m) {
            const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
            const uint64_t word = __ballot(x == v);
            if (lane == 0) planes[static_cast<int64_t>(pid) * W + w] = word;
            ++pid;
            m &= m - 1;
        }
    }
}

__device__ __forceinline__ bool pred_valid(uint32_t label, uint32_t op, uint32_t rsv0, uint32_t rsv1, uint64_t v3,
                                           int32_t L)
{
    return static_cast<int32_t>(label) < L && op <= 2 && rsv0 == 0 && rsv1 == 0 &&
           (op == PC_OP_EXISTS || (v3 >> 63) == 0);
}

// Program entries: plane id, plus flags on the last entry of a clause.
constexpr uint32_t kLast = 1u << 30;
constexpr uint32_t kNeg = 1u << 31;
constexpr uint32_t kPidMask = kLast - 1;
constexpr int32_t kRowFalse = -1;  // some clause admits no node (or a malformed predicate)
constexpr int32_t kRowLong = -2;   // program longer than 4 entries per predicate: decoded on the fly
constexpr int kBatch = 8;          // plane loads in flight per wavefront

__device__ __forceinline__ uint32_t plane_id(const uint64_t *pres, const uint32_t *wb, uint32_t v)
{
    const uint32_t k = v >> 6;
    return wb[k] + __popcll(pres[k] & ((1ull << (v & 63)) - 1));
}

// One thread per row: validate the row and compile it into a clause
// program over plane ids.  A clause is an OR of planes, optionally
// negated; each label value of a node lies in exactly one present plane,
// so In S = OR(S) = NOT OR(present \ S) and NotIn S = NOT OR(S) =
// OR(present \ S): the shorter form is kept.  Entries live at
// prog[4 * pred_off[i] ...], at most 4 per predicate.
__global__ __launch_bounds__(256) void k_sel_compile(const int32_t *__restrict__ pred_off,
                                                     const pc_pred *__restrict__ preds, int64_t n_preds, int32_t I,
                                                     int32_t L, const uint64_t *__restrict__ present,
                                                     const uint32_t *__restrict__ wbase, uint32_t *__restrict__ prog,
                                                     int32_t *__restrict__ row_len, uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < I; i += gridDim.x * blockDim.x) {
        const int64_t b = pred_off[i], e = pred_off[i + 1];
        if (!pc_range_ok(b, e, n_preds)) {
            errs |= PC_DERR_OFFSETS;
            row_len[i] = kRowFalse;
            continue;
        }
        int32_t state = 0;  // 0 ok, kRowFalse, kRowLong
        int64_t n = 0;
        const int64_t cap = 4 * (e - b);
        uint32_t *out = prog + 4 * b;
        for (int64_t p = b; p < e; ++p) {
            const pc_pred q = preds[p];
            if (!pred_valid(q.label, q.op, q.rsv0, q.rsv1, q.vals[3], L)) {
                errs |= PC_DERR_PRED;
                state = kRowFalse;
                continue;
            }
            if (state == kRowFalse) continue;
            const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
            const uint32_t *wb = wbase + static_cast<int64_t>(q.label) * 4;
            uint64_t sel[4];
            bool neg;
            if (q.op == PC_OP_EXISTS) {
                // Exists = NOT OR(plane of the absent value), when any node lacks the label
                sel[0] = sel[1] = sel[2] = 0;
                sel[3] = pres[3] & (1ull << 63);
                neg = true;
            } else {
                uint64_t in[4], out_[4];
                uint32_t ms = 0, mc = 0;
                for (int k = 0; k < 4; ++k) {
                    in[k] = q.vals[k] & pres[k];
                    out_[k] = pres[k] & ~q.vals[k];
                    ms += __popcll(in[k]);
                    mc += __popcll(out_[k]);
                }
                const bool use_in = ms <= mc;
                for (int k = 0; k < 4; ++k) sel[k] = use_in ? in[k] : out_[k];
                neg = (q.op == PC_OP_IN) ? !use_in : use_in;
            }
            uint32_t cnt = __popcll(sel[0]) + __popcll(sel[1]) + __popcll(sel[2]) + __popcll(sel[3]);
            if (cnt == 0) {
                if (!neg) state = kRowFalse;  // empty OR: no node
                continue;                     // negated empty OR: every node
            }
            if (state == kRowLong || n + cnt > cap) {
                state = kRowLong;
                continue;
            }
            for (int k = 0; k < 4; ++k) {
                uint64_t m = sel[k];
                while (m) {
                    const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                    m &= m - 1;
                    uint32_t ent = plane_id(pres, wb, v);
                    if (--cnt == 0) ent |= kLast | (neg ? kNeg : 0u);
                    out[n++] = ent;
                }
            }
        }
        row_len[i] = state ? state : static_cast<int32_t>(n);
    }
    if (errs) atomicOr(d_err, errs);
}

// Rows whose program did not fit: decode the predicates on the scalar unit.
__device__ uint64_t eval_row_decoded(const pc_pred *__restrict__ preds, int64_t b, int64_t e,
                                     const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
                                     const uint64_t *pcol, int32_t W, bool wok)
{
    uint64_t acc = ~0ull;
    for (int64_t p = b; p < e; ++p) {
        const pc_pred *q = preds + p;
        const uint32_t label = q->label, op = q->op;
        const uint64_t *pres = present + static_cast<int64_t>(label) * 4;
        const uint32_t *wb = wbase + static_cast<int64_t>(label) * 4;
        if (op == PC_OP_EXISTS) {
            const uint64_t p3 = pres[3];
            if (p3 >> 63) acc &= wok ? ~pcol[static_cast<int64_t>(plane_id(pres, wb, 255)) * W] : 0ull;
            continue;
        }
        uint64_t cur = 0;
        for (int k = 0; k < 4; ++k) {
            uint64_t m = q->vals[k] & pres[k];
            while (m) {
                const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                m &= m - 1;
                if (wok) cur |= pcol[static_cast<int64_t>(plane_id(pres, wb, v)) * W];
            }
        }
        acc &= (op == PC_OP_IN) ? cur : ~cur;
    }
    return acc;
}

__global__ __launch_bounds__(kEvalThreads) void k_sel_eval(
    const int32_t *__restrict__ pred_off, const pc_pred *__restrict__ preds, int32_t I,
    const uint32_t *__restrict__ prog, const int32_t *__restrict__ row_len, const uint64_t *__restrict__ present,
    const uint32_t *__restrict__ wbase, const uint64_t *__restrict__ planes, int32_t W, int32_t N,
    uint64_t *__restrict__ feasible, uint32_t *__restrict__ popcnt, int32_t ntiles, int32_t nchunks,
    int32_t rows_per_chunk)
{
    const int64_t total = static_cast<int64_t>(ntiles) * nchunks;
    const int64_t item = pc_xcd_item(total);
    if (item >= total) return;
    const int32_t tile = static_cast<int32_t>(item / nchunks);
    const int32_t chunk = static_cast<int32_t>(item % nchunks);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t w = tile * 64 + lane;
    const bool wok = w < W;
    uint64_t tail = ~0ull;
    if (!wok) tail = 0;
    else if (w == W - 1 && (N & 63)) tail = (1ull << (N & 63)) - 1;
    const uint64_t *pcol = planes + (wok ? w : 0);
    const int32_t r0 = chunk * rows_per_chunk;
    const int32_t r1 = min(I, r0 + rows_per_chunk);
    for (int32_t r = r0 + wave; r < r1; r += kEvalThreads / 64) {
        const int32_t len = row_len[r];
        uint64_t acc = ~0ull;
        if (len == kRowFalse) {
            acc = 0;
        } else if (len == kRowLong) {
            acc = eval_row_decoded(preds, pred_off[r], pred_off[r + 1], present, wbase, pcol, W, wok);
        } else {
            const uint32_t *pr = prog + 4 * static_cast<int64_t>(pred_off[r]);
            uint64_t cur = 0;
            for (int32_t e0 = 0; e0 < len; e0 += kBatch) {
                uint32_t E[kBatch];
                uint64_t V[kBatch];
#pragma unroll
                for (int k = 0; k < kBatch; ++k) E[k] = (e0 + k < len) ? pr[e0 + k] : 0u;
#pragma unroll
                for (int k = 0; k < kBatch; ++k)
                    V[k] = (e0 + k < len && wok) ? pcol[static_cast<int64_t>(E[k] & kPidMask) * W] : 0ull;
#pragma unroll
                for (int k = 0; k < kBatch; ++k) {
                    if (e0 + k < len) {
                        cur |= V[k];
                        if (E[k] & kLast) {
                            acc &= (E[k] & kNeg) ? ~cur : cur;
                            cur = 0;
                        }
                    }
                }
                if (__ballot((acc & tail) != 0) == 0) break;
            }
        }
        acc &= tail;
        if (wok) feasible[static_cast<int64_t>(r) * W + w] = acc;
        const uint32_t cnt = pc_wave_sum_u32(__popcll(acc));
        if (lane == 0 && cnt) atomicAdd(&popcnt[r], cnt);
    }
}

}  // namespace

int run_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                  const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                  hipStream_t stream)
{
    const int64_t W = (static_cast<int64_t>(N) + 63) / 64;
    const int64_t pmax = static_cast<int64_t>(L) * (N < 256 ? N : 256);
    const size_t plane_bytes = static_cast<size_t>(pmax) * static_cast<size_t>(W) * 8;
    if (plane_bytes > (size_t(64) << 30))
        return pc_set_error(ctx, PC_ENOMEM, "pc_eval_selectors: value planes need %zu bytes (L=%d N=%d)", plane_bytes,
                            L, N);
    Carver c{nullptr, 0};
    uint64_t *present, *planes;
    uint32_t *wbase, *prog;
    int32_t *row_len;
    auto carve = [&](Carver &cv) {
        present = cv.take<uint64_t>(static_cast<size_t>(L) * 4 + 1);
        wbase = cv.take<uint32_t>(static_cast<size_t>(L) * 4 + 1);
        planes = cv.take<uint64_t>(static_cast<size_t>(pmax) * W + 1);
        prog = cv.take<uint32_t>(static_cast<size_t>(n_preds) * 4 + 1);
        row_len = cv.take<int32_t>(static_cast<size_t>(I) + 1);
    };
    carve(c);
    int rc = pc_ensure_arena(ctx, c.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    launch_fill_u32(popcnt, static_cast<size_t>(I), 0, stream);
    launch_fill_u64(present, static_cast<size_t>(L) * 4, 0, stream);
    PC_LAUNCH_CHECK(ctx);
    if (N > 0 && L > 0) {
        int64_t chunk = kPresenceNodes;
        while ((N + chunk - 1) / chunk > 65535) chunk *= 2;
        dim3 gp((L + 63) / 64, static_cast<unsigned>((N + chunk - 1) / chunk));
        PC_TIMED(ctx, "k_sel_presence", stream, hipLaunchKernelGGL(k_sel_presence, gp, dim3(256), 0, stream, labels, N, L, chunk,
                           reinterpret_cast<uint32_t *>(present)));
        PC_LAUNCH_CHECK(ctx);
    }
    if (L > 0) {
        PC_TIMED(ctx, "k_sel_label_scan", stream, hipLaunchKernelGGL(k_sel_label_scan, dim3(1), dim3(1024), 0, stream, present, L, wbase));
        PC_LAUNCH_CHECK(ctx);
    }
    if (N > 0 && L > 0) {
        dim3 gb(static_cast<unsigned>(W), static_cast<unsigned>((L + 3) / 4));
        PC_TIMED(ctx, "k_sel_planes", stream, hipLaunchKernelGGL(k_sel_planes, gb, dim3(256), 0, stream, labels, N, L, present, wbase, planes,
                           static_cast<int32_t>(W)));
        PC_LAUNCH_CHECK(ctx);
    }
    const int32_t ntiles = static_cast<int32_t>(W > 0 ? (W + 63) / 64 : 1);
    int64_t nchunks = (4096 + ntiles - 1) / ntiles;
    const int64_t max_chunks = (static_cast<int64_t>(I) + 3) / 4;
    if (nchunks > max_chunks) nchunks = max_chunks;
    if (nchunks < 1) nchunks = 1;
    const int32_t rpc = static_cast<int32_t>((I + nchunks - 1) / nchunks);
    nchunks = (I + rpc - 1) / rpc;
    const int64_t total = ntiles * nchunks;
    const unsigned blocks = static_cast<unsigned>(8 * ((total + 7) / 8));
    {
        int64_t cb = (I + 255) / 256;
        if (cb > 8192) cb = 8192;
        PC_TIMED(ctx, "k_sel_compile", stream,
                 hipLaunchKernelGGL(k_sel_compile, dim3(static_cast<unsigned>(cb)), dim3(256), 0, stream, pred_off,
                                    preds, n_preds, I, L, present, wbase, prog, row_len, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    PC_TIMED(ctx, "k_sel_eval", stream,
             hipLaunchKernelGGL(k_sel_eval, dim3(blocks), dim3(kEvalThreads), 0, stream, pred_off, preds, I, prog,
                                row_len, present, wbase, planes, static_cast<int32_t>(W), N, feasible, popcnt,
                                ntiles, static_cast<int32_t>(nchunks), rpc));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

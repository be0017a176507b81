// A5 -- compliant-path existence and hop distance: breadth-first search
// restricted to the switches whose jurisdiction an intent allows.
//
// The paper's path scheduler searches the live topology for a
// constraint-respecting path (weighted Dijkstra with a BFS fallback;
// Network orchestration); as a validator check the question is whether a
// path exists that never leaves the allowed jurisdictions, and how long the
// shortest one is.  Vertex v is allowed for query q iff bit region[v] of
// allowed[q] is set; distances are hop counts in the allowed-induced
// subgraph, -1 when unreachable or when the source is not allowed.
//
// Design (gfx950):
//   bitset : graphs that fit in LDS (27 bytes per vertex): 64 queries per
//            workgroup, one bit each, level-synchronous frontier bitsets
//            (visited / frontier / next) in LDS, push expansion of a
//            compacted frontier list (a few lanes per vertex, coalesced
//            adjacency reads) with 64-bit LDS atomic OR, the per-query
//            allowed mask applied per vertex as a precomputed 64-bit region
//            mask; stops when every query's target is resolved or no
//            frontier bit is left.  The per-vertex words sit in XOR-swizzled
//            slots: vertices 16 apart map to different LDS banks (unswizzled,
//            a fat-tree core's pushes to its per-pod peers, 48 apart, all
//            hit one bank pair).
//   queue  : larger graphs: one workgroup per query, frontier queue in
//            scratch, the distance row itself (or a scratch row, with
//            targets) as the visited set claimed with compare-and-swap.
#include <algorithm>

#include "pc_internal.h"

namespace {

constexpr int kBitsetThreads = 1024;  // two workgroups per CU fill all 32 wave slots
constexpr int kQueueThreads = 256;
constexpr int kMaxBitsetV = 6016;  // 3 x 8 B + 1 B + 2 B per vertex, plus masks, within 160 KB of LDS

__device__ __forceinline__ bool allowed_v(const uint8_t *region, uint32_t A, int32_t v)
{
    const uint32_t r = region[v];
    return r < 32 && ((A >> r) & 1u);
}

// Is v in the forbidden list of one query (Kf entries, -1 = unused)?
__device__ __forceinline__ bool forbidden_v(const int32_t *__restrict__ fl, int32_t Kf, int32_t v)
{
    for (int32_t k = 0; k < Kf; ++k)
        if (fl[k] == v) return true;
    return false;
}

// Waypoint / forbidden lists: every entry must be -1 or a vertex.
__global__ void k_rc_id_check(int64_t n, const int32_t *__restrict__ ids, int32_t V, uint32_t *__restrict__ d_err)
{
    bool bad = false;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int32_t v = ids[i];
        bad |= (v < -1 || v >= V);
    }
    if (bad) atomicOr(d_err, PC_DERR_SWITCH);
}

// *flag stays 1 only if every adjacency list is sorted and every valid
// entry u -> v has its reverse v -> u (a vertex whose offsets are invalid has
// no entries, so no valid list may name it): then the search from v reaches
// u exactly when the search from u reaches v, at the same distance.  One
// wavefront per vertex, its lanes over the vertex's entries.
__global__ __launch_bounds__(256) void k_rc_symcheck(int32_t V, const int32_t *__restrict__ adj_off,
                                                     const int32_t *__restrict__ adj, int64_t n_adj,
                                                     int32_t *__restrict__ flag)
{
    const int lane = threadIdx.x & 63;
    const int32_t waves = gridDim.x * 4;
    bool bad = false;
    for (int32_t u = blockIdx.x * 4 + (threadIdx.x >> 6); u < V; u += waves) {
        const int64_t b = adj_off[u], e = adj_off[u + 1];
        if (!pc_range_ok(b, e, n_adj)) continue;
        for (int64_t p = b + lane; p < e; p += 64) {
            const int32_t v = adj[p];
            if (p > b && adj[p - 1] > v) bad = true;
            if (v < 0 || v >= V) continue;
            int64_t lo = adj_off[v], hi = adj_off[v + 1];
            if (!pc_range_ok(lo, hi, n_adj)) {
                bad = true;
                continue;
            }
            const int64_t end = hi;
            while (lo < hi) {  // first entry >= u
                const int64_t mid = (lo + hi) >> 1;
                if (adj[mid] < u) lo = mid + 1;
                else hi = mid;
            }
            if (lo >= end || adj[lo] != u) bad = true;
        }
    }
    if (__ballot(bad) && lane == 0) atomicAnd(flag, 0);
}

__global__ void k_rc_validate(int32_t V, const int32_t *__restrict__ adj_off, const int32_t *__restrict__ adj,
                              int64_t n_adj, const uint8_t *__restrict__ region, int32_t Q,
                              const int32_t *__restrict__ src, const int32_t *__restrict__ target,
                              uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const int64_t i0 = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
    for (int64_t v = i0; v < V; v += stride) {
        if (region[v] >= 32) errs |= PC_DERR_JUR;
        if (!pc_range_ok(adj_off[v], adj_off[v + 1], n_adj)) errs |= PC_DERR_OFFSETS;
    }
    for (int64_t p = i0; p < n_adj; p += stride) {
        const int32_t v = adj[p];
        if (v < 0 || v >= V) errs |= PC_DERR_GRAPH;
    }
    for (int64_t q = i0; q < Q; q += stride) {
        if (src[q] < 0 || src[q] >= V) errs |= PC_DERR_SWITCH;
        if (target && (target[q] < 0 || target[q] >= V)) errs |= PC_DERR_SWITCH;
    }
    if (errs) atomicOr(d_err, errs);
}

// Append v to an LDS list when `add`, one counter update per wavefront
// (every active lane of the wavefront calls this together).
__device__ __forceinline__ void wave_append(bool add, uint16_t v, int32_t *count, uint16_t *list)
{
    const uint64_t b = __ballot(add);
    if (b == 0) return;
    const int leader = __builtin_ctzll(b);
    const int lane = threadIdx.x & 63;
    int32_t base = 0;
    if (lane == leader) base = atomicAdd(count, static_cast<int32_t>(__popcll(b)));
    base = __shfl(base, leader, 64);
    if (add) {
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(b >> 32),
                                                         __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(b), 0u));
        list[base + static_cast<int32_t>(below)] = v;
    }
}

// Queries ordered by source for the bitset search: a counting sort (the
// order among queries of one source is arbitrary; every result is per
// query).  A workgroup's 64 queries then share few sources, so their
// frontiers overlap and one push along an edge serves many of them.
// Sources outside [0, V) go to bucket V.  Counting: each workgroup ranks its
// queries within their buckets in LDS and reserves its share of every
// bucket it meets with one global atomic (a few thousand instead of one
// per query on the same few counters); pos[q] = the query's place within
// its bucket.
constexpr int kSortThreads = 1024;
constexpr int kSortPer = 4096;  // queries per counting workgroup

__global__ __launch_bounds__(kSortThreads) void k_rc_src_count(int32_t Q, const int32_t *__restrict__ src, int32_t V,
                                                               int32_t *__restrict__ cnt, int32_t *__restrict__ pos)
{
    extern __shared__ int32_t loc[];  // [V + 1] per-bucket counts, then the workgroup's bases
    for (int32_t b = threadIdx.x; b <= V; b += kSortThreads) loc[b] = 0;
    __syncthreads();
    const int32_t q0 = blockIdx.x * kSortPer;
    const int32_t q1 = min(Q, q0 + kSortPer);
    for (int32_t q = q0 + threadIdx.x; q < q1; q += kSortThreads) {
        const int32_t s = src[q];
        pos[q] = atomicAdd(loc + ((s >= 0 && s < V) ? s : V), 1);
    }
    __syncthreads();
    for (int32_t b = threadIdx.x; b <= V; b += kSortThreads) {
        const int32_t n = loc[b];
        loc[b] = n ? atomicAdd(cnt + b, n) : 0;
    }
    __syncthreads();
    for (int32_t q = q0 + threadIdx.x; q < q1; q += kSortThreads) {
        const int32_t s = src[q];
        pos[q] += loc[(s >= 0 && s < V) ? s : V];
    }
}

__global__ void k_rc_src_place(int32_t Q, const int32_t *__restrict__ src, int32_t V, const int32_t *__restrict__ off,
                               const int32_t *__restrict__ pos, int32_t *__restrict__ perm)
{
    for (int32_t q = blockIdx.x * blockDim.x + threadIdx.x; q < Q; q += gridDim.x * blockDim.x) {
        const int32_t s = src[q];
        perm[off[(s >= 0 && s < V) ? s : V] + pos[q]] = q;
    }
}

// 64 queries per workgroup; dist is [Q][V] (target == nullptr) or [Q].
// Each level pushes the frontier along its edges: the frontier vertices are
// kept as a list in LDS and GS lanes share one vertex's adjacency, so the
// adjacency loads are coalesced and the vertex's frontier word is a
// broadcast; the next frontier is built (and the list rewritten) in one
// pass over the vertices.
template <int GS>
__global__ __launch_bounds__(kBitsetThreads) void k_rc_bitset(int32_t V, const int32_t *__restrict__ adj_off,
                                                              const int32_t *__restrict__ adj, int64_t n_adj,
                                                              const uint8_t *__restrict__ region, int32_t Q,
                                                              const int32_t *__restrict__ src,
                                                              const uint32_t *__restrict__ allowed,
                                                              const int32_t *__restrict__ target,
                                                              int32_t *__restrict__ dist,
                                                              const int32_t *__restrict__ forbid, int32_t Kf,
                                                              int32_t qdiv, const int32_t *__restrict__ sym,
                                                              const int32_t *__restrict__ perm)
{
    extern __shared__ uint64_t lds[];
    // visited / frontier / next words of vertex v sit in slot sl(v) =
    // v ^ ((v >> 4) & 15), a permutation of each block of 16, so that
    // vertices a multiple of 16 apart (a core switch's aggregation peers,
    // one per pod) fall in different LDS banks; Vp slots each
    const int32_t Vp = (V + 15) & ~15;
    auto sl = [](int32_t v) { return v ^ ((v >> 4) & 15); };
    uint64_t *vis = lds;
    uint64_t *fr = vis + Vp;
    uint64_t *nx = fr + Vp;
    uint64_t *rmask = nx + Vp;                                              // [32]
    uint8_t *reg = reinterpret_cast<uint8_t *>(rmask + 32);                 // [V]
    uint16_t *flist = reinterpret_cast<uint16_t *>(reg + ((V + 3) & ~3));  // [V] frontier vertices
    __shared__ int32_t nfr[2];                                              // list lengths, by level parity
    __shared__ int flag_done;
    // target look-ahead: the targets' adjacency as (query, entry) pairs
    __shared__ int32_t toff[65], tbeg[64];
    __shared__ unsigned long long found, act;
    // queries still searching (target mode): resolved queries' frontier
    // bits are dropped, so their searches stop spreading
    __shared__ unsigned long long live;
    // query of bit k: qid[k] (queries taken in perm order when given)
    __shared__ int32_t qid[64];
    const int tid = threadIdx.x, lane = tid & 63;
    const int32_t q0 = blockIdx.x * 64;
    const int32_t nq = min(64, Q - q0);
    if (tid < 64) qid[lane] = lane < nq ? (perm ? perm[q0 + lane] : q0 + lane) : 0;
    for (int32_t v = tid; v < Vp; v += kBitsetThreads) {
        vis[v] = 0;
        fr[v] = 0;
        nx[v] = 0;
        if (v < V) reg[v] = region[v];
    }
    if (tid < 64) {
        const uint32_t A = lane < nq ? allowed[qid[lane] / qdiv] : 0u;
        for (int r = 0; r < 32; ++r) {
            const uint64_t m = __ballot((A >> r) & 1u);
            if (lane == 0) rmask[r] = m;
        }
    }
    if (tid == 0) nfr[0] = nfr[1] = 0;
    __syncthreads();
    // forbidden vertices start out visited, so they are never entered
    if (Kf > 0) {
        if (tid < 64 && lane < nq) {
            const int32_t *fl = forbid + static_cast<int64_t>(qid[lane] / qdiv) * Kf;
            for (int32_t k = 0; k < Kf; ++k) {
                const int32_t f = fl[k];
                if (f >= 0 && f < V) atomicOr(reinterpret_cast<unsigned long long *>(&vis[sl(f)]), 1ull << lane);
            }
        }
        __syncthreads();
    }
    // sources; per-query result state lives in wave 0, lane = query
    int32_t res = -1, tgt = -1;
    bool done = true;
    if (tid < 64 && lane < nq) {
        const int32_t q = qid[lane];
        const int32_t s = src[q];
        const bool s_ok = s >= 0 && s < V && allowed_v(reg, allowed[q / qdiv], s) && !((vis[sl(s)] >> lane) & 1);
        if (target) {
            // a target that is not allowed, or forbidden, is never reached:
            // the query is resolved (-1) without a search
            tgt = target[q];
            done = !(s_ok && tgt >= 0 && tgt < V && allowed_v(reg, allowed[q / qdiv], tgt) &&
                     !((vis[sl(tgt)] >> lane) & 1));
        }
        if (s_ok) {
            atomicOr(reinterpret_cast<unsigned long long *>(&fr[sl(s)]), 1ull << lane);
            atomicOr(reinterpret_cast<unsigned long long *>(&vis[sl(s)]), 1ull << lane);
            if (!target) dist[static_cast<int64_t>(q) * V + s] = 0;
        }
    }
    __syncthreads();
    for (int32_t v = tid; v < V; v += kBitsetThreads)
        wave_append(fr[sl(v)] != 0, static_cast<uint16_t>(v), &nfr[0], flist);
    if (tid < 64) {
        if (!done && ((vis[sl(tgt)] >> lane) & 1)) {
            res = 0;
            done = true;
        }
        // A query whose target is allowed and has a neighbour in its
        // frontier at distance d is resolved at d + 1 without expanding
        // that frontier: list each such target's adjacency once.  Only on
        // a symmetric graph (*sym == 1), where the target's list names
        // exactly the vertices whose lists name the target.
        int32_t deg = 0, b = 0;
        bool t_allowed = false;
        if (target && !done && *sym == 1) {
            const int64_t b64 = adj_off[tgt], e64 = adj_off[tgt + 1];
            t_allowed = allowed_v(reg, allowed[qid[lane] / qdiv], tgt);
            if (t_allowed && pc_range_ok(b64, e64, n_adj)) {
                b = static_cast<int32_t>(b64);
                deg = static_cast<int32_t>(e64 - b64);
            }
        }
        int32_t x = deg;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        toff[lane] = x - deg;
        tbeg[lane] = b;
        if (lane == 63) toff[64] = x;
        const uint64_t a = __ballot(deg > 0);
        if (lane == 0) act = a;
        const uint64_t lv = target ? __ballot(!done) : ~0ull;
        if (lane == 0) live = lv;
    }
    __syncthreads();
    const int grp = tid / GS, gl = tid % GS;
    constexpr int kNG = kBitsetThreads / GS;  // groups
    for (int32_t d = 1;; ++d) {
        const int cur = (d - 1) & 1;
        const int32_t nf = nfr[cur];
        if (tid == 0) nfr[cur ^ 1] = 0;  // last read at the start of the previous level
        // A group takes GS frontier entries at a time: lane k loads entry k's
        // adjacency range and frontier word in one round (no dependent load
        // chain per vertex), then the group walks the GS entries, taking
        // each range and word from lane k by shuffle.
        for (int32_t i0 = grp; i0 < nf; i0 += kNG * GS) {
            const int32_t my = i0 + kNG * gl;
            int32_t b = 0, e = 0;
            uint32_t flo = 0, fhi = 0;
            if (my < nf) {
                const int32_t u = flist[my];
                const int64_t b64 = adj_off[u], e64 = adj_off[u + 1];
                if (pc_range_ok(b64, e64, n_adj)) {
                    b = static_cast<int32_t>(b64);
                    e = static_cast<int32_t>(e64);
                    const uint64_t f = fr[sl(u)];
                    flo = static_cast<uint32_t>(f);
                    fhi = static_cast<uint32_t>(f >> 32);
                }
            }
            const int32_t nk = min(GS, (nf - i0 + kNG - 1) / kNG);
            for (int k = 0; k < nk; ++k) {
                const int32_t bk = __shfl(b, k, GS), ek = __shfl(e, k, GS);
                const uint64_t fk = static_cast<uint64_t>(static_cast<uint32_t>(__shfl(fhi, k, GS))) << 32 |
                                    static_cast<uint32_t>(__shfl(flo, k, GS));
                for (int32_t p = bk + gl; p < ek; p += GS) {
                    const int32_t v = adj[p];
                    if (v >= 0 && v < V) atomicOr(reinterpret_cast<unsigned long long *>(&nx[sl(v)]), fk);
                }
            }
        }
        __syncthreads();
        for (int32_t v = tid; v < V; v += kBitsetThreads) {
            const int32_t x = sl(v);
            uint64_t n = nx[x];
            if (n) {
                nx[x] = 0;
                const uint32_t r = reg[v];
                n &= (r < 32 ? rmask[r] : 0ull) & ~vis[x] & live;
                vis[x] |= n;
                if (!target) {
                    uint64_t m = n;
                    while (m) {
                        const int q = __builtin_ctzll(m);
                        m &= m - 1;
                        dist[static_cast<int64_t>(qid[q]) * V + v] = d;
                    }
                }
            }
            fr[x] = n;
            wave_append(n != 0, static_cast<uint16_t>(v), &nfr[cur ^ 1], flist);
        }
        if (tid == 0) found = 0;
        __syncthreads();
        if (target) {
            const uint64_t a = act;
            if (a) {
                const int32_t total = toff[64];
                for (int32_t i = tid; i < total; i += kBitsetThreads) {
                    int32_t lo = 0, hi = 64;  // query q: toff[q] <= i < toff[q + 1]
                    while (hi - lo > 1) {
                        const int32_t mid = (lo + hi) >> 1;
                        if (toff[mid] <= i) lo = mid;
                        else hi = mid;
                    }
                    if (!((a >> lo) & 1)) continue;
                    const int32_t u = adj[tbeg[lo] + (i - toff[lo])];
                    if (u >= 0 && u < V && ((fr[sl(u)] >> lo) & 1)) atomicOr(&found, 1ull << lo);
                }
            }
            __syncthreads();
        }
        if (tid < 64) {
            if (!done && ((fr[sl(tgt)] >> lane) & 1)) {
                res = d;
                done = true;
            } else if (!done && target && ((found >> lane) & 1)) {
                res = d + 1;
                done = true;
            }
            const uint64_t still = __ballot(!done);
            if (tid == 0) {
                flag_done = target ? still == 0 : 0;
                act &= still;
                if (target) live = still;
            }
        }
        __syncthreads();
        // nfr[cur ^ 1] is reset only two levels on; flag_done is rewritten
        // only after the next level's second barrier
        if (nfr[cur ^ 1] == 0 || flag_done) break;
    }
    if (target && tid < 64 && lane < nq) dist[qid[lane]] = res;
}

// One workgroup per query (grid-stride over queries).
__global__ __launch_bounds__(kQueueThreads) void k_rc_queue(int32_t V, const int32_t *__restrict__ adj_off,
                                                            const int32_t *__restrict__ adj, int64_t n_adj,
                                                            const uint8_t *__restrict__ region, int32_t Q,
                                                            const int32_t *__restrict__ src,
                                                            const uint32_t *__restrict__ allowed,
                                                            const int32_t *__restrict__ target,
                                                            int32_t *__restrict__ dist, int32_t *__restrict__ qbuf_all,
                                                            int32_t *__restrict__ rows_all,
                                                            const int32_t *__restrict__ forbid, int32_t Kf,
                                                            int32_t qdiv)
{
    __shared__ int32_t tail_s;
    const int tid = threadIdx.x;
    int32_t *qbuf = qbuf_all + static_cast<int64_t>(blockIdx.x) * V;
    for (int32_t q = blockIdx.x; q < Q; q += gridDim.x) {
        int32_t *drow = target ? rows_all + static_cast<int64_t>(blockIdx.x) * V : dist + static_cast<int64_t>(q) * V;
        const uint32_t A = allowed[q / qdiv];
        const int32_t s = src[q];
        const int32_t tgt = target ? target[q] : -1;
        const int32_t *fl = Kf > 0 ? forbid + static_cast<int64_t>(q / qdiv) * Kf : nullptr;
        const bool s_ok = s >= 0 && s < V && allowed_v(region, A, s) && !forbidden_v(fl, Kf, s);
        // a target that is not allowed, or forbidden, is never reached
        const bool t_ok =
            !target || (tgt >= 0 && tgt < V && allowed_v(region, A, tgt) && !forbidden_v(fl, Kf, tgt));
        if (tid == 0) {
            tail_s = 0;
            if (s_ok && t_ok) {
                drow[s] = 0;
                qbuf[0] = s;
                tail_s = 1;
            }
        }
        __syncthreads();
        int32_t lo = 0, hi = tail_s;
        for (int32_t d = 0; lo < hi; ++d) {
            if (target && t_ok && drow[tgt] != -1) break;
            for (int32_t i = lo + tid; i < hi; i += kQueueThreads) {
                const int32_t u = qbuf[i];
                const int64_t b = adj_off[u], e = adj_off[u + 1];
                if (!pc_range_ok(b, e, n_adj)) continue;
                for (int64_t p = b; p < e; ++p) {
                    const int32_t v = adj[p];
                    if (v < 0 || v >= V || !allowed_v(region, A, v) || forbidden_v(fl, Kf, v)) continue;
                    if (atomicCAS(&drow[v], -1, d + 1) == -1) qbuf[atomicAdd(&tail_s, 1)] = v;
                }
            }
            __syncthreads();
            lo = hi;
            hi = tail_s;
            __syncthreads();
        }
        if (target) {
            __syncthreads();
            if (tid == 0) dist[q] = (s_ok && t_ok) ? drow[tgt] : -1;
            __syncthreads();
            const int32_t n = tail_s;
            for (int32_t i = tid; i < n; i += kQueueThreads) drow[qbuf[i]] = -1;
        }
        __syncthreads();
    }
}

}  // namespace

namespace {

void validate(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
              const uint8_t *region, int32_t Q, const int32_t *src, const int32_t *target, hipStream_t stream)
{
    const int64_t nval = (V > Q ? V : Q) > n_adj ? (V > Q ? V : Q) : n_adj;
    if (nval > 0) {
        int64_t blocks = (nval + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        PC_TIMED(ctx, "k_rc_validate", stream, hipLaunchKernelGGL(k_rc_validate, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, V, adj_off, adj,
                           n_adj, region, Q, src, target, ctx->d_err));
    }
}

// The symmetry flag of the graph, in ctx->d_small[4] (1 = symmetric,
// sorted lists; see k_rc_symcheck).
int32_t *symcheck(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                  hipStream_t stream)
{
    int32_t *sym = ctx->d_small + 4;
    launch_fill_u32(reinterpret_cast<uint32_t *>(sym), 1, 1u, stream);
    if (V > 0)
        PC_TIMED(ctx, "k_rc_symcheck", stream,
                 hipLaunchKernelGGL(k_rc_symcheck, dim3(static_cast<unsigned>(std::min<int64_t>((V + 3) / 4, 8192))),
                                    dim3(256), 0, stream, V, adj_off, adj, n_adj, sym));
    return sym;
}

// BFS of Q queries; query j's allowed mask is allowed[j / qdiv] and its
// forbidden list forbid[(j / qdiv) * Kf ...] (Kf = 0: none).  sym: the
// graph's symmetry flag when the caller has it, else nullptr.  Takes the
// context's arena when it needs scratch.
int bfs(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj, const uint8_t *region,
        int32_t Q, const int32_t *src, const uint32_t *allowed, const int32_t *target, int32_t *dist,
        const int32_t *forbid, int32_t Kf, int32_t qdiv, const int32_t *sym, hipStream_t stream)
{
    if (!target) launch_fill_u32(reinterpret_cast<uint32_t *>(dist), static_cast<size_t>(Q) * V, 0xFFFFFFFFu, stream);
    if (V == 0) {
        if (target) launch_fill_u32(reinterpret_cast<uint32_t *>(dist), static_cast<size_t>(Q), 0xFFFFFFFFu, stream);
        PC_LAUNCH_CHECK(ctx);
        return PC_OK;
    }
    int max_lds = 0;
    PC_HIP(ctx, hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, ctx->device));
    // visited / frontier / next (8 B each), region (1 B) and list (2 B) per vertex
    const size_t lds = ((static_cast<size_t>(V) + 15) & ~size_t(15)) * 3 * 8 + 32 * 8 +
                       ((static_cast<size_t>(V) + 3) & ~size_t(3)) + static_cast<size_t>(V) * 2;
    hipFuncAttributes fa{};
    PC_HIP(ctx, hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(k_rc_bitset<16>)));  // static LDS
    if (V <= kMaxBitsetV && lds + fa.sharedSizeBytes <= static_cast<size_t>(max_lds)) {
        if (!sym && target) sym = symcheck(ctx, V, adj_off, adj, n_adj, stream);
        if (!sym) sym = ctx->d_small + 5;  // full rows: no look-ahead reads it
        PC_LAUNCH_CHECK(ctx);
        // more than one workgroup: order the queries by source
        int32_t *perm = nullptr;
        if (Q > 64) {
            int32_t *cnt, *off, *pos;
            auto carve = [&](Carver &c) {
                cnt = c.take<int32_t>(static_cast<size_t>(V) + 2);
                off = c.take<int32_t>(static_cast<size_t>(V) + 2);
                pos = c.take<int32_t>(static_cast<size_t>(Q));
                perm = c.take<int32_t>(static_cast<size_t>(Q));
            };
            Carver dry{nullptr, 0};
            carve(dry);
            int rc = pc_ensure_arena(ctx, dry.off);
            if (rc) return rc;
            Carver real{ctx->arena, 0};
            carve(real);
            launch_fill_u32(reinterpret_cast<uint32_t *>(cnt), static_cast<size_t>(V) + 1, 0, stream);
            PC_TIMED(ctx, "k_rc_src_count", stream,
                     hipLaunchKernelGGL(k_rc_src_count, dim3(static_cast<unsigned>((Q + kSortPer - 1) / kSortPer)),
                                        dim3(kSortThreads), (static_cast<size_t>(V) + 1) * sizeof(int32_t), stream, Q,
                                        src, V, cnt, pos));
            launch_scan_i32(cnt, V + 1, off, nullptr, nullptr, stream);
            PC_TIMED(ctx, "k_rc_src_place", stream,
                     hipLaunchKernelGGL(k_rc_src_place, dim3(static_cast<unsigned>(std::min<int64_t>((Q + 255) / 256, 4096))),
                                        dim3(256), 0, stream, Q, src, V, off, pos, perm));
            PC_LAUNCH_CHECK(ctx);
        }
        // lanes per vertex: a power of two near a third of the mean degree
        const int64_t avg = n_adj / V;
        const int gs = avg <= 12 ? 4 : avg <= 24 ? 8 : avg <= 48 ? 16 : 32;
        const dim3 grid_b(static_cast<unsigned>((Q + 63) / 64));
        auto launch = [&](auto kern) -> int {
            PC_HIP(ctx, hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
            PC_TIMED(ctx, "k_rc_bitset", stream,
                     hipLaunchKernelGGL(kern, grid_b, dim3(kBitsetThreads), lds, stream, V, adj_off, adj, n_adj,
                                        region, Q, src, allowed, target, dist, forbid, Kf, qdiv, sym, perm));
            PC_LAUNCH_CHECK(ctx);
            return PC_OK;
        };
        if (gs == 4) return launch(k_rc_bitset<4>);
        if (gs == 8) return launch(k_rc_bitset<8>);
        if (gs == 16) return launch(k_rc_bitset<16>);
        return launch(k_rc_bitset<32>);
    }
    int32_t grid = Q < 256 ? Q : 256;
    int32_t *qbuf, *rows;
    auto carve = [&](Carver &c) {
        qbuf = c.take<int32_t>(static_cast<size_t>(grid) * V);
        rows = c.take<int32_t>(target ? static_cast<size_t>(grid) * V : 1);
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);
    if (target) launch_fill_u32(reinterpret_cast<uint32_t *>(rows), static_cast<size_t>(grid) * V, 0xFFFFFFFFu, stream);
    PC_TIMED(ctx, "k_rc_queue", stream, hipLaunchKernelGGL(k_rc_queue, dim3(static_cast<unsigned>(grid)), dim3(kQueueThreads), 0, stream, V, adj_off, adj,
                       n_adj, region, Q, src, allowed, target, dist, qbuf, rows, forbid, Kf, qdiv));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

// Leg k of query q (k <= m, m = waypoints before the first -1) runs from the
// previous waypoint (or src) to the next one (or target); legs past m are
// inactive (src -1).  On a symmetric graph (*sym == 1) legs 0, 2, 4, ... are
// searched from their far end, so that legs 2j and 2j + 1 start at the same
// waypoint and share their frontiers in the workgroup's bitsets.
__global__ void k_rc_legs(int32_t Q, const int32_t *__restrict__ src, const int32_t *__restrict__ target,
                          const int32_t *__restrict__ via, int32_t Kv, const int32_t *__restrict__ sym,
                          int32_t *__restrict__ leg_src, int32_t *__restrict__ leg_tgt)
{
    const bool flip = *sym == 1;
    const int32_t q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= Q) return;
    const int32_t *w = via + static_cast<int64_t>(q) * Kv;
    int32_t *ls = leg_src + static_cast<int64_t>(q) * (Kv + 1);
    int32_t *lt = leg_tgt + static_cast<int64_t>(q) * (Kv + 1);
    int32_t from = src[q];
    bool active = true;
    for (int32_t k = 0; k <= Kv; ++k) {
        const int32_t nxt = k < Kv ? w[k] : -1;
        if (!active) {
            ls[k] = -1;
            lt[k] = -1;
        } else {
            const int32_t to = nxt == -1 ? target[q] : nxt;  // the last leg ends at the target
            const bool rev = flip && (k & 1) == 0;
            ls[k] = rev ? to : from;
            lt[k] = rev ? from : to;
            from = to;
            active = nxt != -1;
        }
    }
}

// dist[q] = sum of the distances of q's active legs, -1 if any is -1
// (saturating at INT32_MAX).
__global__ void k_rc_via_sum(int32_t Q, const int32_t *__restrict__ via, int32_t Kv,
                             const int32_t *__restrict__ leg_dist, int32_t *__restrict__ dist)
{
    const int32_t q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= Q) return;
    const int32_t *w = via + static_cast<int64_t>(q) * Kv;
    const int32_t *ld = leg_dist + static_cast<int64_t>(q) * (Kv + 1);
    int64_t total = 0;
    for (int32_t k = 0; k <= Kv; ++k) {
        const int32_t d = ld[k];
        if (d < 0) {
            total = -1;
            break;
        }
        total += d;
        if (k == Kv || w[k] == -1) break;
    }
    dist[q] = static_cast<int32_t>(total > 0x7FFFFFFF ? 0x7FFFFFFF : total);
}

}  // namespace

int run_reach(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
              const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed, const int32_t *target,
              int32_t *dist, hipStream_t stream)
{
    validate(ctx, V, adj_off, adj, n_adj, region, Q, src, target, stream);
    PC_LAUNCH_CHECK(ctx);
    return bfs(ctx, V, adj_off, adj, n_adj, region, Q, src, allowed, target, dist, nullptr, 0, 1, nullptr, stream);
}

int run_reach_via(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                  const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                  const int32_t *target, const int32_t *via, int32_t Kv, const int32_t *forbid, int32_t Kf,
                  int32_t *dist, hipStream_t stream)
{
    validate(ctx, V, adj_off, adj, n_adj, region, Q, src, target, stream);
    const int64_t nv = static_cast<int64_t>(Q) * Kv, nf = static_cast<int64_t>(Q) * Kf;
    if (nv > 0)
        PC_TIMED(ctx, "k_rc_id_check", stream,
                 hipLaunchKernelGGL(k_rc_id_check, dim3(static_cast<unsigned>(std::min<int64_t>((nv + 255) / 256, 4096))),
                                    dim3(256), 0, stream, nv, via, V, ctx->d_err));
    if (nf > 0)
        PC_TIMED(ctx, "k_rc_id_check", stream,
                 hipLaunchKernelGGL(k_rc_id_check, dim3(static_cast<unsigned>(std::min<int64_t>((nf + 255) / 256, 4096))),
                                    dim3(256), 0, stream, nf, forbid, V, ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    if (Q == 0) return PC_OK;
    if (Kv == 0)
        return bfs(ctx, V, adj_off, adj, n_adj, region, Q, src, allowed, target, dist, forbid, Kf, 1, nullptr,
                   stream);
    // legs [Q][Kv + 1] (sources, targets, distances) in the auxiliary
    // buffer; leg j belongs to query j / (Kv + 1)
    const int64_t nl = static_cast<int64_t>(Q) * (Kv + 1);
    if (nl > 0x7FFFFFFF) return pc_set_error(ctx, PC_EINVAL, "pc_masked_reach_via: Q*(Kv+1) over 2^31 legs");
    int32_t *leg_src, *leg_tgt, *leg_dist;
    auto carve = [&](Carver &c) {
        leg_src = c.take<int32_t>(static_cast<size_t>(nl));
        leg_tgt = c.take<int32_t>(static_cast<size_t>(nl));
        leg_dist = c.take<int32_t>(static_cast<size_t>(nl));
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_aux(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->aux, 0};
    carve(real);
    const unsigned qb = static_cast<unsigned>((Q + 255) / 256);
    const int32_t *sym = symcheck(ctx, V, adj_off, adj, n_adj, stream);
    PC_TIMED(ctx, "k_rc_legs", stream,
             hipLaunchKernelGGL(k_rc_legs, dim3(qb), dim3(256), 0, stream, Q, src, target, via, Kv, sym, leg_src,
                                leg_tgt));
    PC_LAUNCH_CHECK(ctx);
    rc = bfs(ctx, V, adj_off, adj, n_adj, region, static_cast<int32_t>(nl), leg_src, allowed, leg_tgt, leg_dist,
             forbid, Kf, Kv + 1, sym, stream);
    if (rc) return rc;
    PC_TIMED(ctx, "k_rc_via_sum", stream,
             hipLaunchKernelGGL(k_rc_via_sum, dim3(qb), dim3(256), 0, stream, Q, via, Kv, leg_dist, dist));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

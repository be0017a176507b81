// NEXT-2 -- compliant path synthesis: the path scheduler's search for a
// minimum-weight walk through allowed, non-forbidden switches via ordered
// waypoints (weighted Dijkstra, BFS when every link weighs 1), and the
// walk's compilation into one exact-match flow rule per switch (paper,
// Network orchestration).
//
// Design (gfx950):
//   1. validate : the data-error flags, a sweep over the whole input.
//   2. in-links : the reverse of the port graph -- per switch v the (u, port)
//                 pairs of the links u -> v -- counted, scanned and filled.
//   3. search   : one workgroup per request.  Its usable-switch bitset,
//                 distances and frontier queues live in LDS.  Each leg is
//                 a chaotic relaxation in rounds: a wavefront takes 64
//                 frontier switches at a time (one lane each reads the
//                 port range), then relaxes them one after another, its
//                 lanes over a switch's ports with LDS atomic minima,
//                 loading the next switch's links while the current one's
//                 are relaxed; a switch whose distance drops joins the next
//                 round's frontier once (a flag bit per switch).  A frontier switch at or beyond the target's
//                 current distance is skipped: with weights >= 1 it cannot
//                 shorten the target's path, so every switch nearer than
//                 the target ends with its exact distance.  The leg is then
//                 walked back from its end by one wavefront: the
//                 predecessor of v is the lowest-numbered u among v's
//                 in-links with dist(u) + w = dist(v) (a wavefront minimum;
//                 the in-link lists carry each link's weight).
//                 The legs' switches collect in an LDS walk; the rules are
//                 written from it, one wavefront per switch finding the port
//                 of least (weight, index) to the next switch.
#include <climits>

#include "pc_internal.h"

namespace {

constexpr int kPsThreads = 512;  // 8 wavefronts: four such workgroups fit a CU's LDS at fat-tree sizes
constexpr int kPsWaves = kPsThreads / 64;
constexpr int32_t kInf = INT32_MAX;

__device__ __forceinline__ int32_t wave_min_i32(int32_t v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, 64));
    return v;
}

// Data-error flags, each a property of the whole input.
__global__ __launch_bounds__(256) void k_ps_validate(int32_t V, const int32_t *__restrict__ port_off,
                                                     const int32_t *__restrict__ port_peer, int64_t n_ports,
                                                     const uint32_t *__restrict__ weight,
                                                     const uint8_t *__restrict__ region, int32_t Q,
                                                     const int32_t *__restrict__ src,
                                                     const int32_t *__restrict__ target,
                                                     const int32_t *__restrict__ out_port,
                                                     const int32_t *__restrict__ via, int32_t Kv,
                                                     const int32_t *__restrict__ forbid, int32_t Kf,
                                                     uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    const int64_t per_q = Kv > Kf ? (Kv > 1 ? Kv : 1) : (Kf > 1 ? Kf : 1);
    int64_t tot = static_cast<int64_t>(Q) * per_q;
    if (n_ports > tot) tot = n_ports;
    if (V > tot) tot = V;
    for (int64_t x = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; x < tot;
         x += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (x < V) {
            if (region[x] >= 32) errs |= PC_DERR_JUR;
            if (!pc_range_ok(port_off[x], port_off[x + 1], n_ports)) errs |= PC_DERR_OFFSETS;
        }
        if (x < n_ports) {
            if (port_peer[x] < -1 || port_peer[x] >= V) errs |= PC_DERR_SWITCH;
            if (weight && weight[x] == 0) errs |= PC_DERR_GRAPH;
        }
        if (x < Q) {
            const int32_t t = target[x];
            if (src[x] < 0 || src[x] >= V || t < 0 || t >= V) {
                errs |= PC_DERR_SWITCH;
            } else if (pc_range_ok(port_off[t], port_off[t + 1], n_ports) &&
                       (out_port[x] < 0 || out_port[x] >= port_off[t + 1] - port_off[t])) {
                errs |= PC_DERR_ACTION;
            }
        }
        if (x < static_cast<int64_t>(Q) * Kv && (via[x] < -1 || via[x] >= V)) errs |= PC_DERR_SWITCH;
        if (x < static_cast<int64_t>(Q) * Kf && (forbid[x] < -1 || forbid[x] >= V)) errs |= PC_DERR_SWITCH;
    }
    if (errs) atomicOr(d_err, errs);
}

// Weight of port p as a link, or 0 when it is none.
__device__ __forceinline__ uint32_t link_weight(const int32_t *__restrict__ port_peer,
                                                const uint32_t *__restrict__ weight, int32_t V, int64_t p)
{
    const int32_t v = port_peer[p];
    if (v < 0 || v >= V) return 0;
    return weight ? weight[p] : 1u;
}

// In-link counts: one thread per switch u, +1 at the peer of each link.
__global__ __launch_bounds__(256) void k_ps_in_count(int32_t V, const int32_t *__restrict__ port_off,
                                                     const int32_t *__restrict__ port_peer, int64_t n_ports,
                                                     const uint32_t *__restrict__ weight, int32_t *__restrict__ cnt)
{
    const int32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= V) return;
    const int64_t b = port_off[u], e = port_off[u + 1];
    if (!pc_range_ok(b, e, n_ports)) return;
    for (int64_t p = b; p < e; ++p)
        if (link_weight(port_peer, weight, V, p)) atomicAdd(&cnt[port_peer[p]], 1);
}

// In-link lists: (u, link weight) pairs in rin[rin_off[v] ..); cursor starts as a
// copy of rin_off.  The order within a list is arbitrary (only minima are
// taken over it).
__global__ __launch_bounds__(256) void k_ps_in_fill(int32_t V, const int32_t *__restrict__ port_off,
                                                    const int32_t *__restrict__ port_peer, int64_t n_ports,
                                                    const uint32_t *__restrict__ weight,
                                                    int32_t *__restrict__ cursor, int2 *__restrict__ rin)
{
    const int32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= V) return;
    const int64_t b = port_off[u], e = port_off[u + 1];
    if (!pc_range_ok(b, e, n_ports)) return;
    for (int64_t p = b; p < e; ++p) {
        const uint32_t w = link_weight(port_peer, weight, V, p);
        if (w) {
            const int32_t pos = atomicAdd(&cursor[port_peer[p]], 1);
            rin[pos] = make_int2(u, static_cast<int32_t>(w));  // the weight's bits
        }
    }
}

// One workgroup per request (see the file header).  Dynamic LDS: dist,
// two frontier queues (V each), the round flags and the usable bits
// (ceil(V/32) words each), the walk and one leg (max_hops + 2 each).
__global__ __launch_bounds__(kPsThreads) void k_ps_search(
    int32_t V, const int32_t *__restrict__ port_off, const int32_t *__restrict__ port_peer, int64_t n_ports,
    const uint32_t *__restrict__ weight, const uint8_t *__restrict__ region, const int32_t *__restrict__ rin_off,
    const int2 *__restrict__ rin, const int32_t *__restrict__ src, const int32_t *__restrict__ target,
    const uint32_t *__restrict__ allowed, const int32_t *__restrict__ via, int32_t Kv,
    const int32_t *__restrict__ forbid, int32_t Kf, const pc_key *__restrict__ key,
    const int32_t *__restrict__ out_port, int32_t prio, int32_t max_hops, int32_t *__restrict__ hops_out,
    int32_t *__restrict__ path_out, pc_rule *__restrict__ rules_out)
{
    extern __shared__ int32_t ps_lds[];
    const int32_t VW = (V + 31) >> 5;
    int32_t *dist = ps_lds;
    int32_t *qa = dist + V;
    int32_t *qb = qa + V;
    uint32_t *inflag = reinterpret_cast<uint32_t *>(qb + V);
    uint32_t *usable = inflag + VW;
    int32_t *walk = reinterpret_cast<int32_t *>(usable + VW);
    int32_t *leg = walk + max_hops + 2;
    __shared__ int32_t s_nf, s_fail, s_total;

    const int32_t q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t slots = max_hops + 1;
    const int32_t s = src[q], t = target[q];
    bool fail = s < 0 || s >= V || t < 0 || t >= V;
    if (!fail) {
        const int64_t tb = port_off[t], te = port_off[t + 1];
        fail = !pc_range_ok(tb, te, n_ports) || out_port[q] < 0 || out_port[q] >= te - tb;
    }
    const uint32_t A = allowed[q];
    // usable bits: each wavefront takes 64 switches (two words) at a time
    for (int32_t v0 = wave * 64; v0 < V; v0 += kPsWaves * 64) {
        const int32_t v = v0 + lane;
        const uint32_t r = v < V ? region[v] : 32u;
        const uint64_t m = __ballot(r < 32 && ((A >> r) & 1u));
        if (lane < 2 && (v0 >> 5) + lane < VW) usable[(v0 >> 5) + lane] = static_cast<uint32_t>(m >> (32 * lane));
    }
    __syncthreads();
    if (tid < Kf) {
        const int32_t f = forbid[static_cast<int64_t>(q) * Kf + tid];
        if (f >= 0 && f < V) atomicAnd(&usable[f >> 5], ~(1u << (f & 31)));
    }
    if (tid == 0) {
        s_fail = fail;
        s_total = 0;
        if (!fail) walk[0] = s;
    }
    __syncthreads();
    int32_t m = 0;  // waypoints: the list ends at its first -1
    while (m < Kv && via[static_cast<int64_t>(q) * Kv + m] != -1) ++m;
    auto is_usable = [&](int32_t v) { return (usable[v >> 5] >> (v & 31)) & 1u; };

    int32_t from = s;
    for (int32_t li = 0; li <= m && !s_fail; ++li) {
        const int32_t to = li < m ? via[static_cast<int64_t>(q) * Kv + li] : t;
        if (to < 0 || to >= V || !is_usable(from) || !is_usable(to)) break;  // uniform: s_fail set below
        for (int32_t v = tid; v < V; v += kPsThreads) dist[v] = kInf;
        for (int32_t w = tid; w < VW; w += kPsThreads) inflag[w] = 0;
        __syncthreads();
        if (tid == 0) {
            dist[from] = 0;
            qa[0] = from;
            s_nf = 0;
        }
        __syncthreads();
        int32_t nf = 1;
        int32_t *cur = qa, *nxt = qb;
        // Port p's peer and weight: unconditional loads (an index past the
        // switch's last port is clamped to it; the caller drops that lane),
        // whose results nothing touches before relax, so that a wavefront's
        // next switch is fetched while the current one is relaxed.
        const uint32_t *wsrc = weight ? weight : reinterpret_cast<const uint32_t *>(port_peer);
        auto fetch = [&](int64_t p, int64_t e, int32_t &u, uint32_t &w) {
            const int64_t pc = p < e ? p : e - 1;
            u = port_peer[pc];
            w = wsrc[pc];
        };
        // (dto: the target's distance when the switch was taken, an upper
        // bound of the current one, so the pruning stays safe)
        auto relax = [&](int32_t u, uint32_t w, int32_t dv, int32_t dto, int32_t *nxt) {
            if (!weight) w = 1u;
            const bool link = u >= 0 && u < V && w;
            const int32_t uc = link ? u : 0;
            const uint32_t ubits = usable[uc >> 5];  // both LDS reads issued together
            const int32_t du = dist[uc];
            // 32-bit unsigned: distances are below kInf = 2^31 - 1 and a weight
            // of 2^31 - 1 or more cannot shorten any path, so clamping it
            // keeps the sum exact where it matters and below 2^32
            const uint32_t nd32 = static_cast<uint32_t>(dv) + min(w, static_cast<uint32_t>(kInf));
            if (!link || !((ubits >> (uc & 31)) & 1u) || nd32 >= static_cast<uint32_t>(du) ||
                nd32 >= static_cast<uint32_t>(dto))
                return;
            const int32_t nd = static_cast<int32_t>(nd32);
            const int32_t old = atomicMin(&dist[u], nd);
            if (nd < old) {
                const uint32_t bit = 1u << (u & 31);
                if (!(atomicOr(&inflag[u >> 5], bit) & bit)) nxt[atomicAdd(&s_nf, 1)] = u;
            }
        };
        while (nf > 0) {
            // Wavefront `wave` takes frontier entries wave, wave + kPsWaves, ...
            // in batches of 64: each lane reads one entry's port range (one
            // round of loads for 64 switches), then the switches are
            // relaxed one after another, each one's first 64 links loaded
            // while the previous one's are relaxed (two register sets, A
            // and B, in turn).
            for (int32_t base = wave; base < nf; base += kPsWaves * 64) {
                const int32_t idx = base + lane * kPsWaves;
                int32_t vl = 0, bl = 0, el = 0;
                if (idx < nf) {
                    vl = cur[idx];
                    if (dist[vl] < dist[to]) {  // else it cannot shorten the target's path
                        const int32_t b = port_off[vl], e = port_off[vl + 1];
                        if (pc_range_ok(b, e, n_ports)) {
                            bl = b;
                            el = e;
                        }
                    }
                }
                uint64_t live = __ballot(el > bl);
                if (!live) continue;
                // the next switch of the batch (none left: `prev` again, with more = false)
                auto take = [&](int32_t prev, bool &more, int32_t &b, int32_t &e) {
                    more = live != 0;
                    const int32_t jj = more ? static_cast<int32_t>(__builtin_ctzll(live)) : prev;
                    live &= live - 1;
                    b = __builtin_amdgcn_readlane(bl, jj);
                    e = __builtin_amdgcn_readlane(el, jj);
                    return jj;
                };
                auto expand = [&](int32_t jj, int32_t b, int32_t e, int32_t u, uint32_t w) {
                    const int32_t dv = dist[__builtin_amdgcn_readlane(vl, jj)];  // current: it may have dropped
                    const int32_t dto = dist[to];
                    if (static_cast<int64_t>(b) + lane < e) relax(u, w, dv, dto, nxt);
                    for (int64_t p = static_cast<int64_t>(b) + 64 + lane; p < e; p += 64) {
                        int32_t u2;
                        uint32_t w2;
                        fetch(p, e, u2, w2);
                        relax(u2, w2, dv, dto, nxt);
                    }
                };
                bool more;
                int32_t bA, eA, bB, eB, uA, uB;
                uint32_t wA, wB;
                int32_t jA = take(0, more, bA, eA);
                fetch(static_cast<int64_t>(bA) + lane, eA, uA, wA);
                while (true) {
                    const int32_t jB = take(jA, more, bB, eB);
                    fetch(static_cast<int64_t>(bB) + lane, eB, uB, wB);
                    expand(jA, bA, eA, uA, wA);
                    if (!more) break;
                    jA = take(jB, more, bA, eA);
                    fetch(static_cast<int64_t>(bA) + lane, eA, uA, wA);
                    expand(jB, bB, eB, uB, wB);
                    if (!more) break;
                }
            }
            __syncthreads();
            nf = s_nf;
            __syncthreads();
            for (int32_t i = tid; i < nf; i += kPsThreads) {
                const int32_t u = nxt[i];
                atomicAnd(&inflag[u >> 5], ~(1u << (u & 31)));
            }
            if (tid == 0) s_nf = 0;
            int32_t *tmp = cur;
            cur = nxt;
            nxt = tmp;
            __syncthreads();
        }
        if (dist[to] == kInf) break;  // no path: s_fail set below
        if (wave == 0) {
            // walk back from `to`: the lowest-numbered predecessor on a minimum-weight path
            const int32_t total = s_total;
            int32_t c = to, n = 1;
            bool bad = false;
            if (lane == 0) leg[0] = to;
            while (c != from) {
                if (total + n > max_hops) {
                    bad = true;
                    break;
                }
                int32_t best = INT32_MAX;
                const int32_t dc = dist[c];
                for (int32_t k = rin_off[c] + lane; k < rin_off[c + 1]; k += 64) {
                    const int2 in = rin[k];
                    const int32_t du = dist[in.x];
                    if (du != kInf &&
                        static_cast<uint32_t>(du) + min(static_cast<uint32_t>(in.y), static_cast<uint32_t>(kInf)) ==
                            static_cast<uint32_t>(dc))
                        best = min(best, in.x);
                }
                best = wave_min_i32(best);
                if (best == INT32_MAX) {
                    bad = true;
                    break;
                }
                c = best;
                if (lane == 0) leg[n] = c;
                ++n;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (bad) {
                if (lane == 0) s_fail = 1;
            } else {
                for (int32_t i = 1 + lane; i < n; i += 64) walk[total + i] = leg[n - 1 - i];
                if (lane == 0) s_total = total + n - 1;
            }
        }
        __syncthreads();
        from = to;
        if (li == m && !s_fail) from = -1;  // the walk reached the target
    }
    // a leg that broke off before its walk (bad stop or no path) leaves from != -1
    if (tid == 0 && from != -1) s_fail = 1;
    __syncthreads();

    const bool ok = !s_fail;
    const int32_t total = s_total;
    if (tid == 0) hops_out[q] = ok ? total : -1;
    int32_t *pq = path_out + static_cast<int64_t>(q) * slots;
    for (int32_t k = tid; k < slots; k += kPsThreads) pq[k] = (ok && k <= total) ? walk[k] : -1;
    // rules: one wavefront per switch of the walk finds its port to the next switch
    uint32_t *rq = reinterpret_cast<uint32_t *>(rules_out + static_cast<int64_t>(q) * slots);
    for (int32_t k = wave; k < slots; k += kPsWaves) {
        uint32_t action = 0;
        const bool live = ok && k <= total;
        if (live && k < total) {
            const int32_t a = walk[k], bnext = walk[k + 1];
            const int64_t pb = port_off[a], pe = port_off[a + 1];
            uint64_t best = UINT64_MAX;  // (weight << 32) | local port
            for (int64_t p = pb + lane; p < pe; p += 64) {
                const uint32_t w = link_weight(port_peer, weight, V, p);
                if (w && port_peer[p] == bnext) {
                    const uint64_t c = (static_cast<uint64_t>(w) << 32) | static_cast<uint64_t>(p - pb);
                    best = c < best ? c : best;
                }
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                const uint64_t o = __shfl_xor(best, off, 64);
                best = o < best ? o : best;
            }
            action = static_cast<uint32_t>(best & 0xFFFFu);
        } else if (live) {
            action = static_cast<uint32_t>(out_port[q]) & 0xFFFFu;
        }
        // 10 dwords: value[4], mask[4], priority | action << 16, rsv
        if (lane < 10) {
            uint32_t d = 0;
            if (live) {
                if (lane < 4)
                    d = key[q].w[lane];
                else if (lane < 7)
                    d = 0xFFFFFFFFu;
                else if (lane == 7)
                    d = 0xFFu;
                else if (lane == 8)
                    d = static_cast<uint32_t>(prio) | (action << 16);
            }
            rq[static_cast<int64_t>(k) * 10 + lane] = d;
        }
    }
}

}  // namespace

int run_synthesize(pc_ctx *ctx, int32_t V, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                   const uint32_t *weight, const uint8_t *region, int32_t Q, const int32_t *src, const int32_t *target,
                   const uint32_t *allowed, const int32_t *via, int32_t Kv, const int32_t *forbid, int32_t Kf,
                   const pc_key *key, const int32_t *out_port, int32_t prio, int32_t max_hops, int32_t *hops,
                   int32_t *path, pc_rule *rules, hipStream_t stream)
{
    int32_t *cnt, *rin_off, *cursor;
    int2 *rin;
    auto carve = [&](Carver &cv) {
        cnt = cv.take<int32_t>(static_cast<size_t>(V) + 1);
        rin_off = cv.take<int32_t>(static_cast<size_t>(V) + 1);
        cursor = cv.take<int32_t>(static_cast<size_t>(V) + 1);
        rin = cv.take<int2>(static_cast<size_t>(n_ports) + 1);
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    int64_t tot = std::max<int64_t>({static_cast<int64_t>(V), n_ports, static_cast<int64_t>(Q) * std::max(Kv, 1),
                                     static_cast<int64_t>(Q) * std::max(Kf, 1)});
    if (tot > 0) {
        const unsigned g = static_cast<unsigned>(std::min<int64_t>((tot + 255) / 256, 8192));
        PC_TIMED(ctx, "k_ps_validate", stream,
                 hipLaunchKernelGGL(k_ps_validate, dim3(g), dim3(256), 0, stream, V, port_off, port_peer, n_ports,
                                    weight, region, Q, src, target, out_port, via, Kv, forbid, Kf, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (Q == 0) return PC_OK;
    if (V > 0) {
        launch_fill_u32(reinterpret_cast<uint32_t *>(cnt), static_cast<size_t>(V) + 1, 0, stream);
        const unsigned g = static_cast<unsigned>((V + 255) / 256);
        PC_TIMED(ctx, "k_ps_in_count", stream,
                 hipLaunchKernelGGL(k_ps_in_count, dim3(g), dim3(256), 0, stream, V, port_off, port_peer, n_ports,
                                    weight, cnt));
        PC_LAUNCH_CHECK(ctx);
        launch_scan_i32(cnt, V, rin_off, cursor, nullptr, stream);
        PC_LAUNCH_CHECK(ctx);
        PC_TIMED(ctx, "k_ps_in_fill", stream,
                 hipLaunchKernelGGL(k_ps_in_fill, dim3(g), dim3(256), 0, stream, V, port_off, port_peer, n_ports,
                                    weight, cursor, rin));
        PC_LAUNCH_CHECK(ctx);
    }
    const int32_t VW = (V + 31) / 32;
    const size_t lds = (static_cast<size_t>(V) * 3 + static_cast<size_t>(VW) * 2 +
                        2 * static_cast<size_t>(max_hops + 2)) * 4;
    PC_HIP(ctx, hipFuncSetAttribute(reinterpret_cast<const void *>(k_ps_search),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    PC_TIMED(ctx, "k_ps_search", stream,
             hipLaunchKernelGGL(k_ps_search, dim3(static_cast<unsigned>(Q)), dim3(kPsThreads), lds, stream, V,
                                port_off, port_peer, n_ports, weight, region, rin_off, rin, src, target, allowed, via,
                                Kv, forbid, Kf, key, out_port, prio, max_hops, hops, path, rules));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

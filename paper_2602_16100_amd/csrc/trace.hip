// A2-A4 -- routing constraints on the realised paths: trace every header
// hop by hop through the per-switch, priority-ordered ternary flow tables
// and collect the jurisdictions visited.
//
// The paper compiles every path into one flow rule per hop (Network
// orchestration), and a routing constraint is judged on the paths those
// rules actually realise (Formal Model and Satisfaction, condition (ii)); the
// validator checks that realised paths avoid forbidden switches (validator
// check definition).  The first-match rule order (larger priority, then
// lower index), table miss, drop, egress and TTL are the readings written in
// include/pc.h.
//
// Design (gfx950):
//   prep   : per switch, kChunks 4-bit chunks of the 104-bit key chosen from
//            a sample of its rules and of the headers (the chunks on which
//            its rules discriminate most among the headers seen); per
//            32-rule group, for each chunk and each of the 16 chunk values,
//            the 32-bit set of rules whose mask/value admit that value (per-
//            rule admit sets from an LDS table, then a bit transpose across
//            the half-wavefront).  Stored plane-major per switch so a
//            wavefront loads 64 groups with coalesced reads.  Also validates
//            ports, jurisdictions, offsets and actions (the data-error sweep).
//   levels : level-synchronous walk.  Live traces are bucketed by their
//            current switch: a plan pass scans the per-switch counts, a
//            scatter pass writes each trace's 32-byte bucket record (trace,
//            jurisdiction mask, header) at its switch's offset plus its
//            rank.  One workgroup per work item (a switch and a balanced
//            share of its bucket) keeps the switch's chunk sets in VGPRs
//            (8,192 rules per 4-wave slice) and filters every lookup with
//            kChunks uniform-index register reads and ANDs; the rare
//            survivors are verified against the full 104-bit rule and the
//            first match is the minimum of (0xFFFF - priority, index) over
//            the workgroup (LDS 64-bit atomic min).  The same workgroup then
//            applies the match with the switch's ports staged in LDS, counts
//            the moving traces per forwarding port (one count update per
//            port and workgroup, which also gives each trace its rank in its
//            next switch's bucket) and writes their live-list entries in its
//            own share of the list, grouped by port.
//   tail   : once few traces are left in flight, one workgroup per trace
//            walks it to its end, reading only the chunk-set words its
//            header selects.
#include <stdlib.h>

#include <algorithm>

#include "pc_internal.h"

namespace {

constexpr int kChunks = 6;                 // 4-bit chunks of the key used by the filter (chosen per switch)
constexpr int kKeyNibbles = 26;            // the 104-bit key: 8 nibbles in each of w0..w2, 2 in w3's low byte
constexpr int kChooseSample = 512;         // rules per switch sampled to choose its filter chunks
constexpr int kPlaneWords = kChunks * 16;  // words per 32-rule group
constexpr int kMatchWaves = 4;
constexpr int kMatchThreads = kMatchWaves * 64;
constexpr int kSliceGroups = kMatchThreads;  // one group (32 rules) per lane
constexpr int kChunk = 256;                  // lookups per lookup stream of a small table's work item (a multiple of 4)
constexpr int kMaxChunk = 256;               // lookups per work item at most (<= kMatchThreads)
constexpr int kItemCap = 192;                // lookups per work item of a table of kSliceGroups groups or more
constexpr int kQueue = 512;                  // queued filter survivors per wavefront (>= 4 x 64)
constexpr int kPrepGroups = 128;             // groups per prep workgroup (16 wavefronts x 4 rounds x 2 groups)
constexpr uint64_t kNoMatch = ~0ull;
static_assert(kItemCap % 4 == 0 && kItemCap <= kChunk, "an item holds >= kItemCap lookups unless it is its switch's only one");
static_assert(kChunk % 4 == 0 && kMaxChunk % kChunk == 0 && kMaxChunk <= kMatchThreads,
              "one epilogue thread per lookup");
constexpr int kCountPad = 32;  // live-trace counters are 128 bytes apart: contended atomics on one line serialise
constexpr int kPortSlots = 64;  // forwarding ports whose moves a match workgroup counts in LDS

// 16 chunk-value sets of one 4-bit chunk, kept in VGPRs; indexed with a
// wave-uniform value this lowers to register-indexed moves (s_set_gpr_idx).
typedef uint32_t v16u __attribute__((ext_vector_type(16)));

// Bit k set iff slot k of trace t's watch list names switch s (K = 0: none).
__device__ __forceinline__ uint32_t watch_bits(const int32_t *__restrict__ watch, int32_t K, int32_t t, int32_t s)
{
    uint32_t m = 0;
    const int32_t *w = watch + static_cast<int64_t>(t) * K;
    for (int32_t k = 0; k < K; ++k)
        if (w[k] == s) m |= 1u << k;
    return m;
}

// Nibble n (0..25) of a 104-bit key or mask: bits 4(n mod 8) .. +3 of word n / 8.
__device__ __forceinline__ uint32_t key_nibble(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, uint32_t n)
{
    const uint32_t w = n < 8 ? w0 : n < 16 ? w1 : n < 24 ? w2 : w3;
    return (w >> ((n & 7u) * 4u)) & 15u;
}

// Filter chunk c of a switch whose chunk positions are packed in cp (5 bits each).
__device__ __forceinline__ uint32_t chunk_pos(uint32_t cp, int c) { return (cp >> (5 * c)) & 31u; }

// Bit of switch s in a visited-switch summary.
__device__ __forceinline__ uint64_t sum_bit(int32_t s) { return 1ull << (s & 63); }

constexpr int kWalkSlots = 8;  // walk records: the first 8 switches of a walk

__device__ __forceinline__ uint32_t jur_bit(const uint8_t *jur, int32_t s)
{
    const uint32_t j = jur[s];
    return j < 32 ? (1u << j) : 0u;
}

// Per switch: validate offsets / jurisdiction, count 32-rule groups and prep blocks.
__global__ void k_tr_switch_info(int32_t S, const int32_t *__restrict__ port_off, int64_t n_ports,
                                 const uint8_t *__restrict__ jur, const int32_t *__restrict__ rule_off,
                                 int64_t n_rules, int32_t *__restrict__ gcount, int32_t *__restrict__ bcount,
                                 uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    for (int32_t s = blockIdx.x * blockDim.x + threadIdx.x; s < S; s += gridDim.x * blockDim.x) {
        if (jur[s] >= 32) errs |= PC_DERR_JUR;
        const bool pok = pc_range_ok(port_off[s], port_off[s + 1], n_ports);
        const int64_t rb = rule_off[s], re = rule_off[s + 1];
        const bool rok = pc_range_ok(rb, re, n_rules);
        if (!pok || !rok) errs |= PC_DERR_OFFSETS;
        const int64_t g = rok ? (re - rb + 31) / 32 : 0;
        gcount[s] = static_cast<int32_t>(g);
        bcount[s] = static_cast<int32_t>((g + kPrepGroups - 1) / kPrepGroups);
    }
    if (errs) atomicOr(d_err, errs);
}

__global__ void k_tr_port_check(int64_t n_ports, const int32_t *__restrict__ port_peer, int32_t S,
                                uint32_t *__restrict__ d_err)
{
    bool bad = false;
    for (int64_t p = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; p < n_ports;
         p += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int32_t v = port_peer[p];
        bad |= (v < -1 || v >= S);
    }
    if (bad) atomicOr(d_err, PC_DERR_SWITCH);
}

// Per port: its peer and the peer's jurisdiction bit (0 unless the peer is a
// switch), read by the match with one load per port.
__global__ void k_tr_port_info(int64_t n_ports, const int32_t *__restrict__ port_peer, int32_t S,
                               const uint8_t *__restrict__ jur, int2 *__restrict__ pinfo)
{
    for (int64_t p = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; p < n_ports;
         p += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int32_t v = port_peer[p];
        const uint32_t j = v >= 0 && v < S ? jur[v] : 32u;
        pinfo[p] = make_int2(v, j < 32 ? static_cast<int32_t>(1u << j) : 0);
    }
}

// Histogram of the headers' nibble values over a strided sample of at most
// kHeaderSample headers: hh[n][x] = sampled headers whose nibble n is x.
// hh must be zero on entry.
constexpr int kHeaderSample = 65536;
__global__ __launch_bounds__(256) void k_tr_hdr_hist(const pc_key *__restrict__ hdr, int32_t T,
                                                     uint32_t *__restrict__ hh)
{
    __shared__ uint32_t loc[kKeyNibbles * 16];
    for (int i = threadIdx.x; i < kKeyNibbles * 16; i += 256) loc[i] = 0;
    __syncthreads();
    const int64_t stride = T > kHeaderSample ? (static_cast<int64_t>(T) + kHeaderSample - 1) / kHeaderSample : 1;
    for (int64_t i = blockIdx.x * 256 + threadIdx.x; i * stride < T; i += static_cast<int64_t>(gridDim.x) * 256) {
        const pc_key h = hdr[i * stride];
        for (uint32_t n = 0; n < kKeyNibbles; ++n)
            atomicAdd(&loc[n * 16 + key_nibble(h.w[0], h.w[1], h.w[2], h.w[3], n)], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kKeyNibbles * 16; i += 256)
        if (loc[i]) atomicAdd(hh + i, loc[i]);
}

// The filter chunks of each switch (one workgroup per switch).  From a
// sample of at most kChooseSample of its rules (every ceil(R / sample)-th):
// for each of the key's 26 nibbles and each chunk value x, the number A[x]
// of sampled rules whose value/mask admit x.  With hh the headers' nibble
// histogram, score = sum_x (hh[x] + 1) A[x] is proportional to the chance
// that a header drawn like the traced ones (smoothed towards uniform)
// passes the nibble's filter against a rule drawn like the switch's.  The
// kChunks nibbles of smallest score (ties: lower nibble) filter out the
// most: nibbles the rules wildcard, or where headers and rules agree on a
// few values, score high.  Any choice gives the same results; it only
// decides how many rules reach the full 104-bit check.
__global__ __launch_bounds__(256) void k_tr_choose(int32_t S, const int32_t *__restrict__ rule_off, int64_t n_rules,
                                                   const pc_rule *__restrict__ rules,
                                                   const uint32_t *__restrict__ hh, uint32_t *__restrict__ cpos)
{
    __shared__ uint32_t hist[kKeyNibbles][256];  // (value & mask, mask) patterns per nibble
    __shared__ unsigned long long score[kKeyNibbles];
    const int32_t s = blockIdx.x;
    if (s >= S) return;
    for (int i = threadIdx.x; i < kKeyNibbles * 256; i += 256) (&hist[0][0])[i] = 0;
    if (threadIdx.x < kKeyNibbles) score[threadIdx.x] = 0;
    __syncthreads();
    const int64_t rb = rule_off[s], re = rule_off[s + 1];
    const int64_t R = pc_range_ok(rb, re, n_rules) ? re - rb : 0;
    const int64_t stride = R > kChooseSample ? (R + kChooseSample - 1) / kChooseSample : 1;
    for (int64_t i = threadIdx.x; i * stride < R && i < kChooseSample; i += 256) {
        const pc_rule *r = rules + rb + i * stride;
        const uint32_t v0 = r->value.w[0], v1 = r->value.w[1], v2 = r->value.w[2], v3 = r->value.w[3];
        const uint32_t m0 = r->mask.w[0], m1 = r->mask.w[1], m2 = r->mask.w[2], m3 = r->mask.w[3];
        for (uint32_t n = 0; n < kKeyNibbles; ++n) {
            const uint32_t m = key_nibble(m0, m1, m2, m3, n);
            const uint32_t v = key_nibble(v0, v1, v2, v3, n) & m;
            atomicAdd(&hist[n][m << 4 | v], 1u);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kKeyNibbles * 16; i += 256) {
        const int n = i >> 4;
        const uint32_t x = i & 15;
        uint64_t a = 0;  // sampled rules admitting chunk value x: (x & m) == (v & m)
        for (uint32_t m = 0; m < 16; ++m) a += hist[n][m << 4 | (x & m)];
        atomicAdd(&score[n], static_cast<unsigned long long>(a * (static_cast<uint64_t>(hh[n * 16 + x]) + 1)));
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t taken = 0, cp = 0;
        for (int c = 0; c < kChunks; ++c) {
            int best = -1;
            for (int n = 0; n < kKeyNibbles; ++n)
                if (!((taken >> n) & 1u) && (best < 0 || score[n] < score[best])) best = n;
            taken |= 1u << best;
            cp |= static_cast<uint32_t>(best) << (5 * c);
        }
        cpos[s] = cp;
    }
}

// Rows r of a 32-lane half hold 32-bit words x_r; afterwards lane i holds
// column i (bit r = bit i of the old x_r).  Five block-swap stages, one per
// lane-index bit j: the partner's word (lane i ^ j) is rotated so that its
// blocks land where this lane takes them, then merged under the lane's keep
// mask.  The stages commute; each costs one cross-lane move and two VALU ops.
template <int J>
__device__ __forceinline__ uint32_t lane_xor(uint32_t x)
{
    const int v = static_cast<int>(x);
    if constexpr (J == 1) return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
    if constexpr (J == 2) return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
    if constexpr (J == 4) {
        // banks 0 and 2 of each row read lane + 4 (row_shl:4), banks 1 and 3 read lane - 4 (row_shr:4)
        const int lo = __builtin_amdgcn_update_dpp(v, v, 0x104, 0xF, 0x5, false);
        return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(lo, v, 0x114, 0xF, 0xA, false));
    }
    if constexpr (J == 8) return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0x128, 0xF, 0xF, false));  // row_ror:8
    if constexpr (J == 16) return static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(v, 0x401F));  // 32-lane groups, xor 16
    return x;
}

template <int J>
__device__ __forceinline__ uint32_t swap_stage(uint32_t x, uint32_t keep, uint32_t rot)
{
    const uint32_t y = lane_xor<J>(x);
    const uint32_t t = __builtin_amdgcn_alignbit(y, y, rot);  // rotate right
    return (x & keep) | (t & ~keep);
}

__device__ __forceinline__ uint32_t transpose32(uint32_t x, const uint32_t (&keep)[5], const uint32_t (&rot)[5])
{
    x = swap_stage<1>(x, keep[0], rot[0]);
    x = swap_stage<2>(x, keep[1], rot[1]);
    x = swap_stage<4>(x, keep[2], rot[2]);
    x = swap_stage<8>(x, keep[3], rot[3]);
    return swap_stage<16>(x, keep[4], rot[4]);
}

constexpr int kPrepWaves = 16;
constexpr int kPrepRounds = 4;                          // 64-rule rounds per wavefront, loads issued up front
constexpr int kTileStride = kPrepGroups + 2;            // LDS row pitch (spreads a half-wave's rows over banks)
static_assert(kPrepGroups == 2 * kPrepWaves * kPrepRounds, "two groups per wavefront round");

// Build the chunk sets of kPrepGroups groups of one switch; validate actions.
// Lane r of a half-wave holds rule r of a group and looks up, for each chunk,
// the 16-bit set of chunk values its value/mask admit (a 256-entry LDS table
// indexed by the chunk's value & mask and mask).  Two chunks share a word;
// a 32 x 32 bit transpose over the half-wave turns the rules' admit sets
// into the group's per-value rule sets: word (chunk c, value x) lands in lane
// (c % 2) * 16 + x of the transpose of word c / 2.
__global__ __launch_bounds__(1024) void k_tr_prep(int32_t S, const int32_t *__restrict__ port_off, int64_t n_ports,
                                                  const int32_t *__restrict__ rule_off,
                                                  const pc_rule *__restrict__ rules,
                                                  const int32_t *__restrict__ gcount,
                                                  const int32_t *__restrict__ gofs, const int32_t *__restrict__ bofs,
                                                  uint32_t *__restrict__ filt, uint32_t *__restrict__ d_err,
                                                  const uint32_t *__restrict__ only, uint32_t *__restrict__ sw_bad,
                                                  const uint32_t *__restrict__ cpos)
{
    __shared__ uint32_t tile[kPlaneWords * kTileStride];
    __shared__ uint16_t admit[256];
    const int32_t b = blockIdx.x;
    if (b >= bofs[S]) return;
    // switch owning this block: largest s with bofs[s] <= b
    int32_t lo = 0, hi = S;  // invariant: bofs[lo] <= b < bofs[hi]
    while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (bofs[mid] <= b) lo = mid;
        else hi = mid;
    }
    const int32_t s = lo;
    if (only != nullptr && !((only[s >> 5] >> (s & 31)) & 1u)) return;  // only the listed switches (whole block)
    const int32_t G = gcount[s];
    const int32_t g0 = (b - bofs[s]) * kPrepGroups;
    const int64_t rb = rule_off[s];
    const int64_t R = rule_off[s + 1] - rb;
    const bool pok = pc_range_ok(port_off[s], port_off[s + 1], n_ports);
    const int64_t np = pok ? port_off[s + 1] - port_off[s] : 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t cp = cpos[s];
    // issue every round's loads before any use
    uint4 vv[kPrepRounds], mm[kPrepRounds];
    uint32_t act[kPrepRounds];
    bool ok[kPrepRounds];
#pragma unroll
    for (int k = 0; k < kPrepRounds; ++k) {
        const int32_t gl = 2 * (wave * kPrepRounds + k) + (lane >> 5);
        const int64_t local = static_cast<int64_t>(g0 + gl - (lane >> 5)) * 32 + lane;  // rule index within the switch
        ok[k] = local < R && g0 + gl < G;
        vv[k] = mm[k] = make_uint4(0, 0, 0, 0);
        act[k] = 0;
        if (ok[k]) {
            const pc_rule *r = rules + rb + local;
            vv[k] = make_uint4(r->value.w[0], r->value.w[1], r->value.w[2], r->value.w[3]);
            mm[k] = make_uint4(r->mask.w[0], r->mask.w[1], r->mask.w[2], r->mask.w[3]);
            act[k] = r->action;
        }
    }
    // admit[(v & m) | m << 4] = set of 4-bit values y with (y & m) == (v & m)
    if (threadIdx.x < 256) {
        const uint32_t m = threadIdx.x >> 4, t = threadIdx.x & 15;
        uint32_t set = 0;
        for (uint32_t y = 0; y < 16; ++y) set |= static_cast<uint32_t>((y & m) == t) << y;
        admit[threadIdx.x] = static_cast<uint16_t>(set);
    }
    // per-stage keep masks and rotations of this lane (stage j = 1, 2, 4, 8, 16)
    uint32_t keep[5], rot[5];
    {
        const uint32_t blk[5] = {0x55555555u, 0x33333333u, 0x0F0F0F0Fu, 0x00FF00FFu, 0x0000FFFFu};
#pragma unroll
        for (int q = 0; q < 5; ++q) {
            const bool up = (lane >> q) & 1;
            keep[q] = up ? ~blk[q] : blk[q];
            rot[q] = up ? (1u << q) : 32u - (1u << q);
        }
    }
    __syncthreads();
    bool bad_action = false;
#pragma unroll
    for (int k = 0; k < kPrepRounds; ++k) {
        uint32_t w[kChunks / 2];
#pragma unroll
        for (int d = 0; d < kChunks / 2; ++d) {
            const uint32_t n0 = chunk_pos(cp, 2 * d), n1 = chunk_pos(cp, 2 * d + 1);
            const uint32_t ma = key_nibble(mm[k].x, mm[k].y, mm[k].z, mm[k].w, n0);
            const uint32_t mb = key_nibble(mm[k].x, mm[k].y, mm[k].z, mm[k].w, n1);
            const uint32_t i0 = (key_nibble(vv[k].x, vv[k].y, vv[k].z, vv[k].w, n0) & ma) | (ma << 4);
            const uint32_t i1 = (key_nibble(vv[k].x, vv[k].y, vv[k].z, vv[k].w, n1) & mb) | (mb << 4);
            const uint32_t a0 = ok[k] ? admit[i0] : 0u, a1 = ok[k] ? admit[i1] : 0u;
            w[d] = transpose32(a0 | (a1 << 16), keep, rot);
        }
        bad_action |= ok[k] && act[k] != PC_ACTION_DROP && static_cast<int64_t>(act[k]) >= np;
        const int gl = 2 * (wave * kPrepRounds + k) + (lane >> 5);
#pragma unroll
        for (int d = 0; d < kChunks / 2; ++d) tile[(32 * d + (lane & 31)) * kTileStride + gl] = w[d];
    }
    if (__ballot(bad_action) && lane == 0) {
        atomicOr(d_err, PC_DERR_ACTION);
        if (sw_bad != nullptr) atomicOr(sw_bad + s, 1u);
    }
    __syncthreads();
    uint32_t *dst = filt + static_cast<int64_t>(gofs[s]) * kPlaneWords;
    for (int i = threadIdx.x; i < kPlaneWords * kPrepGroups; i += blockDim.x) {
        const int row = i / kPrepGroups, gl = i % kPrepGroups;
        const int32_t g = g0 + gl;
        if (g < G) dst[static_cast<int64_t>(row) * G + g] = tile[row * kTileStride + gl];
    }
}

// Level 0: every trace starts at its ingress switch (an invalid ingress
// ends it at once as MISS).  A workgroup takes kInitPer traces, kInitPer /
// 1024 per thread: with kLds (S small enough) it counts them per switch in
// LDS and reserves each switch's share with one global count update, a
// trace's rank being that share's base plus its rank in the workgroup;
// otherwise every trace updates its switch's count itself.  Live-list slots
// are reserved once per workgroup.
// A bucketed lookup: the trace, its jurisdiction mask so far and its
// header, gathered when the trace is bucketed so that the match stages its
// lookups with contiguous loads.
struct __align__(16) BRec {
    int32_t t;
    uint32_t jm;
    uint32_t pad[2];
    pc_key key;
};

// A live-list entry: a trace in flight, the switch it is at, its rank in
// that switch's bucket, its jurisdiction mask so far and its header (next
// = -1: the slot of a trace that has ended).
struct __align__(16) LRec {
    int32_t t;
    int32_t next;
    int32_t rk;
    uint32_t jm;
    pc_key key;
};

constexpr int kInitThreads = 1024;
constexpr int kInitRounds = 4;
constexpr int kInitPer = kInitThreads * kInitRounds;
constexpr int kInitLdsS = 8192;  // switches counted in LDS at most (32 KB)
template <bool kLds>
__global__ __launch_bounds__(kInitThreads) void k_tr_init(int32_t S, const uint8_t *__restrict__ jur,
                                                          const int32_t *__restrict__ ingress,
                                                          const pc_key *__restrict__ hdr, int32_t T,
                                                          LRec *__restrict__ live,
                                                          int32_t *__restrict__ nlive,
                                                          int32_t *__restrict__ counts, pc_trace_out *__restrict__ out,
                                                          const int32_t *__restrict__ watch, int32_t K,
                                                          uint32_t *__restrict__ visit, uint64_t *__restrict__ vsum,
                                                          int32_t *__restrict__ walk, uint32_t *__restrict__ d_err)
{
    extern __shared__ int32_t lcnt[];  // [S] with kLds
    __shared__ int32_t nloc, base;
    if (threadIdx.x == 0) nloc = 0;
    if constexpr (kLds)
        for (int32_t b = threadIdx.x; b < S; b += kInitThreads) lcnt[b] = 0;
    __syncthreads();
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kInitPer;
    int32_t sw[kInitRounds], rk[kInitRounds], slot[kInitRounds];
    uint32_t jb[kInitRounds];
    bool bad = false;
#pragma unroll
    for (int k = 0; k < kInitRounds; ++k) {
        const int64_t t64 = t0 + k * kInitThreads + threadIdx.x;
        const int32_t t = static_cast<int32_t>(t64);
        sw[k] = -1;
        rk[k] = 0;
        jb[k] = 0;
        if (t64 < T) {
            const int32_t s = ingress[t];
            if (s < 0 || s >= S) {
                bad = true;
                pc_trace_out o;
                o.jmask = 0;
                o.last_switch = s;
                o.last_port = PC_NO_PORT;
                o.hops = 0;
                o.state = PC_MISS;
                out[t] = o;
                if (visit) visit[t] = 0;
                if (vsum) vsum[t] = 0;
                if (walk)
                    for (int j = 0; j < kWalkSlots; ++j) walk[static_cast<int64_t>(t) * kWalkSlots + j] = -1;
            } else {
                jb[k] = jur_bit(jur, s);
                if (visit) visit[t] = watch_bits(watch, K, t, s);
                if (vsum) vsum[t] = sum_bit(s);
                if (walk)
                    for (int j = 0; j < kWalkSlots; ++j) walk[static_cast<int64_t>(t) * kWalkSlots + j] = j ? -1 : s;
                sw[k] = s;
                if constexpr (kLds) rk[k] = atomicAdd(&lcnt[s], 1);
                else rk[k] = atomicAdd(&counts[static_cast<int64_t>(s) * kCountPad], 1);
            }
        }
        // a slot in the workgroup's share of the live list: one LDS update per wavefront
        const uint64_t m = __ballot(sw[k] >= 0);
        int32_t wb = 0;
        if ((threadIdx.x & 63) == 0 && m) wb = atomicAdd(&nloc, static_cast<int32_t>(__popcll(m)));
        wb = __shfl(wb, 0, 64);
        slot[k] = sw[k] >= 0 ? wb + static_cast<int32_t>(__builtin_amdgcn_mbcnt_hi(
                                        static_cast<uint32_t>(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)))
                             : -1;
    }
    __syncthreads();
    if constexpr (kLds)
        for (int32_t b = threadIdx.x; b < S; b += kInitThreads) {
            const int32_t n = lcnt[b];
            lcnt[b] = n ? atomicAdd(&counts[static_cast<int64_t>(b) * kCountPad], n) : 0;
        }
    if (threadIdx.x == 0) base = nloc ? atomicAdd(nlive, nloc) : 0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kInitRounds; ++k)
        if (slot[k] >= 0) {
            const int32_t t = static_cast<int32_t>(t0 + k * kInitThreads + threadIdx.x);
            LRec e;
            e.t = t;
            e.next = sw[k];
            e.rk = kLds ? lcnt[sw[k]] + rk[k] : rk[k];
            e.jm = jb[k];
            e.key = hdr[t];
            live[base + slot[k]] = e;
        }
    if (__ballot(bad) && (threadIdx.x & 63) == 0) atomicOr(d_err, PC_DERR_SWITCH);
}

// Bucket the live traces by current switch: a live entry puts its trace at
// slot boff[switch] + rank, its rank having been taken when it was counted.
// The list holds *len entries; traces that ended leave entries with switch
// -1.  Also maps each match work item to (its switch, its index among the
// switch's items): the switch is the last s with ioff[s] <= item.
__global__ void k_tr_scatter(const LRec *__restrict__ live, const int32_t *__restrict__ len, int32_t T, int32_t S,
                             const int32_t *__restrict__ boff, BRec *__restrict__ bucket,
                             const int32_t *__restrict__ ioff, int2 *__restrict__ imap, int32_t icap)
{
    const int32_t n_items = min(ioff[S], icap);
    for (int32_t it = blockIdx.x * blockDim.x + threadIdx.x; it < n_items; it += gridDim.x * blockDim.x) {
        int32_t lo = 0, hi = S;
        while (hi - lo > 1) {
            const int32_t mid = (lo + hi) >> 1;
            if (ioff[mid] <= it) lo = mid;
            else hi = mid;
        }
        imap[it] = make_int2(lo, it - ioff[lo]);
    }
    const int32_t n = min(*len, T);
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int4 e = reinterpret_cast<const int4 *>(live)[2 * i];  // (t, next, rk, jm)
        if (e.y < 0 || e.y >= S || static_cast<uint32_t>(e.x) >= static_cast<uint32_t>(T)) continue;
        const int32_t pos = boff[e.y] + e.z;
        if (pos >= 0 && pos < T) {
            BRec r;
            r.t = e.x;
            r.jm = static_cast<uint32_t>(e.w);
            r.pad[0] = r.pad[1] = 0;
            r.key = live[i].key;
            bucket[pos] = r;
        }
    }
}

__device__ __forceinline__ bool rule_matches(const pc_rule *r, uint32_t h0, uint32_t h1, uint32_t h2, uint32_t h3)
{
    return (((h0 ^ r->value.w[0]) & r->mask.w[0]) | ((h1 ^ r->value.w[1]) & r->mask.w[1]) |
            ((h2 ^ r->value.w[2]) & r->mask.w[2]) | ((h3 ^ r->value.w[3]) & r->mask.w[3])) == 0;
}

// First-match key of a rule: (0xFFFF - priority) << 48 | local index << 16 |
// action.  The smallest key is the highest priority, ties to the lower
// index; the action rides along, so applying the match reads no rule.
__device__ __forceinline__ uint64_t rule_key(const pc_rule *r, uint32_t local)
{
    return (static_cast<uint64_t>(0xFFFFu - r->priority) << 48) | (static_cast<uint64_t>(local) << 16) | r->action;
}

// Verify the surviving rules of one 32-rule group against the full header
// and fold their (priority, index) keys into *best.
__device__ __forceinline__ void verify_group(uint32_t surv, const pc_rule *grp, uint32_t local0, const pc_key &h,
                                             unsigned long long *best)
{
    while (surv) {
        const int bit = __builtin_ctz(surv);
        surv &= surv - 1;
        const pc_rule *r = grp + bit;
        if (rule_matches(r, h.w[0], h.w[1], h.w[2], h.w[3]))
            atomicMin(best, static_cast<unsigned long long>(rule_key(r, local0 + bit)));
    }
}

// Apply the chosen rule (its key, see rule_key) at a switch of np ports (np
// < 0: the switch's port range is invalid) whose port a leads to
// peer_of(a): returns the terminal state, or -1 when the trace moves on to
// *next through port *port.
template <class PeerOf>
__device__ __forceinline__ int apply_key(int32_t S, int32_t ttl, int64_t np, const PeerOf &peer_of, uint64_t key,
                                         int32_t hops, int32_t *next, uint16_t *port)
{
    if (key == kNoMatch) return PC_MISS;
    const uint32_t a = static_cast<uint32_t>(key & 0xFFFFu);
    if (a == PC_ACTION_DROP) return PC_DROP;
    if (np < 0 || static_cast<int64_t>(a) >= np) return PC_MISS;
    const int32_t peer = peer_of(a);
    if (peer == -1) {
        *port = static_cast<uint16_t>(a);
        return PC_EGRESS;
    }
    if (peer < -1 || peer >= S) return PC_MISS;
    if (hops == ttl) return PC_TTL;
    *next = peer;
    *port = static_cast<uint16_t>(a);  // the forwarding port
    return -1;
}

// The same, with switch s's ports read from port_off / port_peer.
__device__ __forceinline__ int apply_rule(int32_t S, const int32_t *__restrict__ port_off,
                                          const int32_t *__restrict__ port_peer, int64_t n_ports, int32_t ttl,
                                          int32_t s, uint64_t key, int32_t hops, int32_t *next, uint16_t *port)
{
    const int64_t pb = port_off[s], pe = port_off[s + 1];
    const int64_t np = pc_range_ok(pb, pe, n_ports) ? pe - pb : -1;
    return apply_key(S, ttl, np, [&](uint32_t a) { return port_peer[pb + a]; }, key, hops, next, port);
}

__device__ __forceinline__ void write_out(pc_trace_out *out, int32_t t, uint32_t jm, int32_t s, uint16_t port,
                                          int32_t hops, int state)
{
    pc_trace_out o;
    o.jmask = jm;
    o.last_switch = s;
    o.last_port = port;
    o.hops = static_cast<uint8_t>(hops);
    o.state = static_cast<uint8_t>(state);
    out[t] = o;
}

// Per-trace state of the level loop and where a level's results go.
struct Level {
    int32_t S;
    int32_t T;              // capacity of the live list
    const int32_t *port_off;
    const int32_t *port_peer;
    const int2 *pinfo;      // per port: (peer, the peer's jurisdiction bit)
    int64_t n_ports;
    const uint8_t *jur;
    int32_t ttl;
    int32_t hops;           // hops every trace of this level has made (the level's index)
    LRec *live_next;        // one entry per lookup of this level, at its bucket slot (switch -1: the trace ended)
    int32_t *nlive_next;    // traces in flight after this level
    int32_t *counts_next;   // live traces per switch after this level
    pc_trace_out *out;
    const int32_t *watch;   // [T][K] switches whose visit is recorded
    int32_t K;
    uint32_t *visit;        // [T] or nullptr
    uint64_t *vsum;         // [T] visited-switch summaries or nullptr
    int32_t *walk;          // [T][kWalkSlots] walk records or nullptr
};

// Lookups per match work item of a switch of G groups with n lookups in
// this level: the switch's lookups split evenly (in multiples of 4) over as
// few items as hold at most kItemCap each, where a table of fewer than
// kSliceGroups groups, which leaves wavefronts free for further lookup
// streams, takes kChunk per stream (at most kMaxChunk).
__device__ __forceinline__ int32_t item_lookups(int32_t G, int32_t n)
{
    const int32_t gws = G >= kSliceGroups ? kMatchWaves : max(1, (G + 63) / 64);
    const int32_t cap = gws == kMatchWaves ? kItemCap : min(kMaxChunk, kChunk * (kMatchWaves / gws));
    const int32_t items = max(1, (n + cap - 1) / cap);
    return max(4, ((n + items - 1) / items + 3) & ~3);
}

// Per level: bucket offsets boff = exclusive scan of counts (which are
// cleared for reuse), work-item offsets ioff = exclusive scan of
// ceil(counts / item_lookups(G, counts)), *total = the level's lookups (the
// length of the live list its match writes), and *nlive_next = 0 for the
// match to count the traces that move on.  One workgroup of 1024 threads;
// each thread takes kPlanPer consecutive switches per pass, so a pass
// covers 4,096 switches with all of its loads in flight together.
constexpr int kPlanPer = 4;
__global__ __launch_bounds__(1024) void k_tr_plan(int32_t *__restrict__ counts, int32_t S, int32_t *__restrict__ boff,
                                                  int32_t *__restrict__ ioff, const int32_t *__restrict__ gcount,
                                                  int32_t *__restrict__ total, int32_t *__restrict__ nlive_next)
{
    __shared__ int32_t wsum[2][16];
    __shared__ int32_t carry_s[2];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    if (tid < 2) carry_s[tid] = 0;
    if (tid == 0) *nlive_next = 0;
    __syncthreads();
    for (int32_t base = 0; base < S; base += 1024 * kPlanPer) {
        const int32_t i0 = base + tid * kPlanPer;
        int32_t v0[kPlanPer], g[kPlanPer], v1[kPlanPer];
#pragma unroll
        for (int k = 0; k < kPlanPer; ++k) {
            v0[k] = i0 + k < S ? counts[static_cast<int64_t>(i0 + k) * kCountPad] : 0;
            g[k] = i0 + k < S ? gcount[i0 + k] : 0;
        }
        int32_t s0 = 0, s1 = 0;
#pragma unroll
        for (int k = 0; k < kPlanPer; ++k) {
            const int32_t ch = item_lookups(g[k], v0[k]);
            v1[k] = (v0[k] + ch - 1) / ch;
            s0 += v0[k];
            s1 += v1[k];
        }
        int32_t x0 = s0, x1 = s1;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t y0 = __shfl_up(x0, off, 64), y1 = __shfl_up(x1, off, 64);
            if (lane >= off) {
                x0 += y0;
                x1 += y1;
            }
        }
        if (lane == 63) {
            wsum[0][wid] = x0;
            wsum[1][wid] = x1;
        }
        __syncthreads();
        if (wid < 2) {
            int32_t w = lane < 16 ? wsum[wid][lane] : 0;
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                const int32_t y = __shfl_up(w, off, 64);
                if (lane >= off) w += y;
            }
            if (lane < 16) wsum[wid][lane] = w;
        }
        __syncthreads();
        const int32_t c0 = carry_s[0], c1 = carry_s[1];
        int32_t e0 = c0 + (wid ? wsum[0][wid - 1] : 0) + x0 - s0;
        int32_t e1 = c1 + (wid ? wsum[1][wid - 1] : 0) + x1 - s1;
#pragma unroll
        for (int k = 0; k < kPlanPer; ++k)
            if (i0 + k < S) {
                boff[i0 + k] = e0;
                ioff[i0 + k] = e1;
                counts[static_cast<int64_t>(i0 + k) * kCountPad] = 0;
                e0 += v0[k];
                e1 += v1[k];
            }
        __syncthreads();
        if (tid == 0) {
            carry_s[0] = c0 + wsum[0][15];
            carry_s[1] = c1 + wsum[1][15];
        }
        __syncthreads();
    }
    if (tid == 0) {
        boff[S] = carry_s[0];
        ioff[S] = carry_s[1];
        *total = carry_s[0];
    }
}

// Filter four lookups: sv[k] = AND over the six chunks c of F[c][x[c][k]].
// GPR index mode stays on while only its index changes, and every indexed
// read feeds its lookup's AND directly; the four lookups' ANDs alternate, so
// consecutive vector instructions do not depend on each other.  The chunk
// sets sit in fixed registers v32..v127 (chunk c at v[32 + 16c .. 47 + 16c]);
// indices are below 16, so every indexed read stays inside its chunk's
// sixteen registers.  Two blocks of three chunks keep the operand lists short.
// Index mode keeps its index in M0, which each block declares clobbered.
#define PC_IDX(a, b, c, d, base, op)                        \
    "s_set_gpr_idx_idx %" #a "\n\t"                          \
    "v_" op "_b32 %0, v" #base ", %0\n\t"                    \
    "s_set_gpr_idx_idx %" #b "\n\t"                          \
    "v_" op "_b32 %1, v" #base ", %1\n\t"                    \
    "s_set_gpr_idx_idx %" #c "\n\t"                          \
    "v_" op "_b32 %2, v" #base ", %2\n\t"                    \
    "s_set_gpr_idx_idx %" #d "\n\t"                          \
    "v_" op "_b32 %3, v" #base ", %3\n\t"
__device__ __forceinline__ void filter_quad(const uint32_t (&x)[kChunks][4], const v16u (&F)[kChunks],
                                            uint32_t (&sv)[4])
{
    uint32_t a0, a1, a2, a3;
    asm volatile(
        "s_set_gpr_idx_on %4, gpr_idx(SRC0)\n\t"
        "v_mov_b32 %0, v32\n\t"
        "s_set_gpr_idx_idx %5\n\t"
        "v_mov_b32 %1, v32\n\t"
        "s_set_gpr_idx_idx %6\n\t"
        "v_mov_b32 %2, v32\n\t"
        "s_set_gpr_idx_idx %7\n\t"
        "v_mov_b32 %3, v32\n\t"
        PC_IDX(8, 9, 10, 11, 48, "and")
        PC_IDX(12, 13, 14, 15, 64, "and")
        "s_set_gpr_idx_off"
        : "=&v"(a0), "=&v"(a1), "=&v"(a2), "=&v"(a3)
        : "s"(x[0][0]), "s"(x[0][1]), "s"(x[0][2]), "s"(x[0][3]), "s"(x[1][0]), "s"(x[1][1]), "s"(x[1][2]),
          "s"(x[1][3]), "s"(x[2][0]), "s"(x[2][1]), "s"(x[2][2]), "s"(x[2][3]), "{v[32:47]}"(F[0]),
          "{v[48:63]}"(F[1]), "{v[64:79]}"(F[2])
        : "m0");
    asm volatile(
        "s_set_gpr_idx_on %4, gpr_idx(SRC0)\n\t"
        "v_and_b32 %0, v80, %0\n\t"
        "s_set_gpr_idx_idx %5\n\t"
        "v_and_b32 %1, v80, %1\n\t"
        "s_set_gpr_idx_idx %6\n\t"
        "v_and_b32 %2, v80, %2\n\t"
        "s_set_gpr_idx_idx %7\n\t"
        "v_and_b32 %3, v80, %3\n\t"
        PC_IDX(8, 9, 10, 11, 96, "and")
        PC_IDX(12, 13, 14, 15, 112, "and")
        "s_set_gpr_idx_off"
        : "+v"(a0), "+v"(a1), "+v"(a2), "+v"(a3)
        : "s"(x[3][0]), "s"(x[3][1]), "s"(x[3][2]), "s"(x[3][3]), "s"(x[4][0]), "s"(x[4][1]), "s"(x[4][2]),
          "s"(x[4][3]), "s"(x[5][0]), "s"(x[5][1]), "s"(x[5][2]), "s"(x[5][3]), "{v[80:95]}"(F[3]),
          "{v[96:111]}"(F[4]), "{v[112:127]}"(F[5])
        : "m0");
    sv[0] = a0;
    sv[1] = a1;
    sv[2] = a2;
    sv[3] = a3;
}
#undef PC_IDX

// One workgroup per work item = (switch, chunk of at most item_lookups(G, n)
// lookups of its bucket).  Items are dealt to XCDs in contiguous ranges, so
// the chunks of one switch share an L2.
__global__ __launch_bounds__(kMatchThreads, 4) void k_tr_match(
    int32_t S, const int32_t *__restrict__ rule_off, const pc_rule *__restrict__ rules,
    const int32_t *__restrict__ gcount, const int32_t *__restrict__ gofs, const uint32_t *__restrict__ filt,
    const int32_t *__restrict__ boff, const int32_t *__restrict__ ioff, const int2 *__restrict__ imap,
    const BRec *__restrict__ bucket, const uint32_t *__restrict__ cpos, Level lv)
{
    __shared__ uint64_t best[kMaxChunk];
    __shared__ __align__(16) uint32_t cidx[kChunks][kMaxChunk];  // each lookup's values of the switch's filter chunks
    __shared__ __align__(16) pc_key keys[kMaxChunk];
    __shared__ int32_t tids[kMaxChunk];
    __shared__ uint32_t tjm[kMaxChunk];  // each lookup's trace: jurisdiction mask so far
    __shared__ uint2 queue[kMatchWaves][kQueue];  // per wavefront: (survivor set, lookup << 6 | lane)
    // the switch's first kPortSlots ports: peer, the peer's jurisdiction
    // bit, and the item's traces that leave through the port (count, then
    // the base of their ranks in the peer's bucket)
    __shared__ int32_t ppeer[kPortSlots], pcnt[kPortSlots], pbase[kPortSlots];
    __shared__ uint32_t pjb[kPortSlots];
    // the item's live entries are ordered by forwarding port: port p's run
    // starts at prun[p], the run of the other ports at prun[kPortSlots]
    __shared__ int32_t prun[kPortSlots + 1];
    __shared__ int32_t nother, nmove;  // traces leaving through the other ports; all that move on
    // the grid was sized from an upper bound on the item count: blocks past
    // the real count's per-XCD share return at once
    const int32_t n_items = ioff[S];
    const int32_t per = (n_items + 7) / 8;
    const int32_t kx = static_cast<int32_t>(blockIdx.x >> 3);
    if (kx >= per) return;
    const int32_t item = static_cast<int32_t>(blockIdx.x & 7) * per + kx;
    if (item >= n_items) return;
    // the item's switch and its index among the switch's items
    const int2 im = imap[item];
    const int32_t s = im.x;
    if (static_cast<uint32_t>(s) >= static_cast<uint32_t>(S)) return;
    const int32_t chunk = item_lookups(gcount[s], boff[s + 1] - boff[s]);
    const int32_t bb = boff[s] + im.y * chunk;
    const int32_t tn = min(chunk, min(boff[s + 1], lv.T) - bb);  // bucket holds at most T entries
    if (tn <= 0) return;
    const int32_t tn4 = (tn + 3) & ~3;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t G = gcount[s];
    const int64_t rb = rule_off[s];
    const uint32_t *fs = filt + static_cast<int64_t>(gofs[s]) * kPlaneWords;
    const int32_t nslices = max(1, (G + kSliceGroups - 1) / kSliceGroups);
    const uint32_t cp = cpos[s];
    uint2 *q = queue[wave];
    // A table of fewer than kSliceGroups groups fills gws wavefronts; the
    // workgroup's other wavefronts take further shares of the lookups: wave
    // = stream * gws + gwi holds groups gwi * 64 .. and filters the lookups
    // of its stream (contiguous quads).  Waves past the last stream idle.
    const int32_t gws = G >= kSliceGroups ? kMatchWaves : max(1, (G + 63) / 64);
    const int32_t streams = kMatchWaves / gws;
    const int32_t gwi = wave % gws, st = wave / gws;
    const int32_t nquads = tn4 / 4;
    const int32_t per_stream = (nquads + streams - 1) / streams;
    const int32_t jb = st < streams ? min(tn4, 4 * st * per_stream) : tn4;
    const int32_t je = st < streams ? min(tn4, 4 * (st + 1) * per_stream) : tn4;
    // the switch's ports (np < 0: its port range is invalid)
    const int64_t pb = lv.port_off[s], pe = lv.port_off[s + 1];
    const int64_t np = pc_range_ok(pb, pe, lv.n_ports) ? pe - pb : -1;
    // A lane's chunk sets of group g: buffer loads with the lane's group as
    // the vector offset (clamped into the table) and the plane as a scalar
    // offset; an opaque copy of the plane stride keeps the 96 offsets from
    // being hoisted out of the loops (and spilled) as invariants.  A lane past
    // the last group gets empty chunk sets, so it never survives the filter;
    // a switch without rules (G = 0) reads offset 0 of an empty buffer, which
    // returns zeros.
    auto load_sets = [&](int32_t g, v16u (&F)[kChunks]) {
        uint32_t pstride = static_cast<uint32_t>(G) * 4u;
        asm volatile("" : "+s"(pstride));
        const __amdgpu_buffer_rsrc_t frs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint32_t *>(fs), static_cast<short>(0), kPlaneWords * G * 4, 0x00020000);
        const uint32_t voff = static_cast<uint32_t>(max(0, min(g, G - 1))) * 4u;
#pragma unroll
        for (int c = 0; c < kChunks; ++c)
#pragma unroll
            for (int x = 0; x < 16; ++x)
                F[c][x] = __builtin_amdgcn_raw_buffer_load_b32(frs, voff, static_cast<uint32_t>(c * 16 + x) * pstride, 0);
        if (g >= G) {
#pragma unroll
            for (int x = 0; x < 16; ++x) F[0][x] = 0u;
        }
    };
    // stage the chunk (at most one lookup per thread: tn4 <= kMaxChunk <=
    // kMatchThreads); pad to a multiple of 4 lookups with copies of the last
    const int i = static_cast<int>(threadIdx.x);
    BRec r{};
    if (i < tn4) r = bucket[bb + min(i, tn - 1)];
    // the first slice's chunk sets load while the lookups are staged
    // (whether or not this wavefront filters: the loads are clamped into the
    // table, and a branch would leave the sets undefined on one path)
    v16u F0[kChunks];
    load_sets(gwi * 64 + lane, F0);
    if (i < tn4) {
        int32_t t = r.t;
        pc_key h = r.key;
        uint32_t jmv = r.jm;
        if (static_cast<uint32_t>(t) >= static_cast<uint32_t>(lv.T)) {  // not a trace id: skipped
            t = -1;
            h = pc_key{};
            jmv = 0;
        }
        tids[i] = t;
        keys[i] = h;
        tjm[i] = jmv;
        best[i] = kNoMatch;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) cidx[c][i] = key_nibble(h.w[0], h.w[1], h.w[2], h.w[3], chunk_pos(cp, c));
    }
    if (threadIdx.x < kPortSlots) {
        const int2 pi = static_cast<int64_t>(threadIdx.x) < np ? lv.pinfo[pb + threadIdx.x] : make_int2(-2, 0);
        ppeer[threadIdx.x] = pi.x;
        pjb[threadIdx.x] = static_cast<uint32_t>(pi.y);
        pcnt[threadIdx.x] = 0;
        if (threadIdx.x == 0) nother = 0;
    }
    __syncthreads();
    // Filter phase: survivors of the chunk filter are queued (per wavefront)
    // until the queue could overflow.  Verify phase: the queued survivors are
    // checked against their full rules, 64 at a time, with the chunk sets
    // dead.  Then filtering resumes with the sets loaded again.  A quad of
    // lookups queues at most 256 entries, so every round advances.  gw is
    // the group of lane 0.
    auto round = [&](int32_t gw, int32_t &jr, const v16u (&F)[kChunks]) {
        int32_t qn = 0;
        int32_t j0 = jr;
        for (; j0 < je; j0 += 4) {
            uint4 X[kChunks];
#pragma unroll
            for (int c = 0; c < kChunks; ++c) X[c] = reinterpret_cast<const uint4 *>(cidx[c])[j0 >> 2];
            uint32_t sv[4];
            uint32_t xi[kChunks][4];
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                xi[c][0] = __builtin_amdgcn_readfirstlane(X[c].x);
                xi[c][1] = __builtin_amdgcn_readfirstlane(X[c].y);
                xi[c][2] = __builtin_amdgcn_readfirstlane(X[c].z);
                xi[c][3] = __builtin_amdgcn_readfirstlane(X[c].w);
            }
            filter_quad(xi, F, sv);
            if (__ballot((sv[0] | sv[1] | sv[2] | sv[3]) != 0)) {
                uint64_t m[4];
                int32_t n = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    m[k] = __ballot(sv[k] != 0);
                    n += __popcll(m[k]);
                }
                if (qn + n > kQueue) break;  // resume at this quad after verifying
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    if (sv[k]) {
                        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
                            static_cast<uint32_t>(m[k] >> 32),
                            __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m[k]), 0u));
                        q[qn + below] = make_uint2(sv[k], static_cast<uint32_t>(j0 + k) << 6 | lane);
                    }
                    qn += __popcll(m[k]);
                }
            }
        }
        jr = j0;
        // the queue entries were written by other lanes of this wavefront
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (int32_t e = lane; e < qn; e += 64) {
            const uint2 en = q[e];
            const int32_t j = static_cast<int32_t>(en.y >> 6);
            const int32_t gg = gw + static_cast<int32_t>(en.y & 63u);
            verify_group(en.x, rules + rb + static_cast<int64_t>(gg) * 32, static_cast<uint32_t>(gg) * 32,
                         keys[j], reinterpret_cast<unsigned long long *>(&best[j]));
        }
        __builtin_amdgcn_wave_barrier();
    };
    // one slice of kSliceGroups groups at a time, one group per lane, its
    // chunk sets held in VGPRs while the chunk's lookups stream past.  The
    // first round of the first slice uses the sets loaded with the staging;
    // it runs outside the slice loop, so those sets are dead after it and
    // never live beside a later round's (inside the loop they would be, and
    // the 192 registers would spill)
    int32_t jr0 = jb;
    if (jb < je) round(gwi * 64, jr0, F0);
    for (int32_t sl = 0; sl < nslices; ++sl) {
        const int32_t g = sl * kSliceGroups + gwi * 64 + lane;
        const int32_t gw = sl * kSliceGroups + gwi * 64;
        int32_t jr = sl == 0 ? jr0 : jb;
        while (jr < je) {
            v16u F[kChunks];
            load_sets(g, F);
            round(gw, jr, F);
        }
    }
    // every wavefront's matches are in best[] (a lookup's matches come from
    // the wavefronts that hold its groups, its epilogue thread may be another)
    __syncthreads();
    // apply the first match.  A trace that moves on is counted in its next
    // switch's bucket (one count update per forwarding port and workgroup;
    // its rank there is the port's base plus its rank in the item) and gets
    // an entry in the item's share of the live list, grouped by port so that
    // the bucketing pass writes runs; the slots after the item's moving
    // traces are marked as ended (switch -1).
    const int32_t h = lv.hops;
    int32_t t = -1, lrank = -1, orank = -1, next = -1, rk = 0;
    uint32_t jm_next = 0;
    uint16_t port = PC_NO_PORT;
    if (threadIdx.x < tn) {  // tn <= kMaxChunk <= kMatchThreads
        t = tids[threadIdx.x];
        if (t >= 0) {
            const uint32_t jmv = tjm[threadIdx.x];
            const int state = apply_key(
                lv.S, lv.ttl, np,
                [&](uint32_t a) { return a < kPortSlots ? ppeer[a] : lv.port_peer[pb + a]; },
                best[threadIdx.x], h, &next, &port);
            if (state >= 0) {
                write_out(lv.out, t, jmv, s, port, h, state);
                t = -1;
            } else {
                jm_next = jmv | (port < kPortSlots ? pjb[port] : jur_bit(lv.jur, next));
                if (lv.visit) lv.visit[t] |= watch_bits(lv.watch, lv.K, t, next);
                if (lv.vsum) lv.vsum[t] |= sum_bit(next);
                if (lv.walk && h + 1 < kWalkSlots) lv.walk[static_cast<int64_t>(t) * kWalkSlots + h + 1] = next;
                if (port < kPortSlots) {
                    lrank = atomicAdd(&pcnt[port], 1);
                } else {
                    rk = atomicAdd(&lv.counts_next[static_cast<int64_t>(next) * kCountPad], 1);
                    orank = atomicAdd(&nother, 1);
                }
            }
        }
    }
    __syncthreads();
    static_assert(kPortSlots == 64, "one wavefront scans the port counts");
    if (threadIdx.x < kPortSlots) {
        const int32_t c = pcnt[threadIdx.x];
        // a port some trace forwarded through: its peer is a valid switch
        if (c > 0) pbase[threadIdx.x] = atomicAdd(&lv.counts_next[static_cast<int64_t>(ppeer[threadIdx.x]) * kCountPad], c);
        int32_t x = c;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        prun[threadIdx.x] = x - c;
        if (threadIdx.x == kPortSlots - 1) {
            prun[kPortSlots] = x;
            const int32_t m = x + nother;
            nmove = m;
            if (m) atomicAdd(lv.nlive_next, m);  // the traces in flight after this level
        }
    }
    __syncthreads();
    int32_t slot = -1;
    if (lrank >= 0) {
        rk = pbase[port] + lrank;
        slot = prun[port] + lrank;
    } else if (orank >= 0) {
        slot = prun[kPortSlots] + orank;
    }
    if (slot >= 0) {
        LRec e;
        e.t = t;
        e.next = next;
        e.rk = rk;
        e.jm = jm_next;
        e.key = keys[threadIdx.x];
        lv.live_next[bb + slot] = e;
    }
    if (threadIdx.x >= nmove && threadIdx.x < tn)
        *reinterpret_cast<int4 *>(lv.live_next + bb + threadIdx.x) = make_int4(-1, -1, 0, 0);
}

// Sparse tail: one workgroup per trace still in flight walks it to its end,
// filtering each switch's rule groups with only the kChunks chunk-set words
// its header selects (coalesced over groups) and reducing the first match in
// LDS.
__global__ __launch_bounds__(256) void k_tr_walk(int32_t S, const int32_t *__restrict__ port_off,
                                                 const int32_t *__restrict__ port_peer, int64_t n_ports,
                                                 const uint8_t *__restrict__ jur, const int32_t *__restrict__ rule_off,
                                                 const pc_rule *__restrict__ rules, const int32_t *__restrict__ gcount,
                                                 const int32_t *__restrict__ gofs, const uint32_t *__restrict__ filt,
                                                 int32_t ttl,
                                                 const LRec *__restrict__ live, const int32_t *__restrict__ len,
                                                 int32_t hops0, pc_trace_out *__restrict__ out,
                                                 const int32_t *__restrict__ watch, int32_t K,
                                                 uint32_t *__restrict__ visit, uint64_t *__restrict__ vsum,
                                                 int32_t *__restrict__ walk, const uint32_t *__restrict__ cpos)
{
    __shared__ unsigned long long best;
    const int32_t n = *len;
    for (int32_t i = blockIdx.x; i < n; i += gridDim.x) {
        const LRec e = live[i];
        if (e.next < 0 || e.next >= S) continue;  // the slot of a trace that has ended
        const int32_t t = e.t;
        const pc_key h = e.key;
        int32_t s = e.next;
        uint32_t jm = e.jm;
        uint32_t vis = visit ? visit[t] : 0u;
        uint64_t vs = vsum ? vsum[t] : 0ull;
        int32_t hops = hops0;
        for (;;) {
            if (threadIdx.x == 0) best = kNoMatch;
            __syncthreads();
            const int32_t G = gcount[s];
            const uint32_t *fs = filt + static_cast<int64_t>(gofs[s]) * kPlaneWords;
            const int64_t rb = rule_off[s];
            const uint32_t cp = cpos[s];
            uint32_t x[kChunks];
#pragma unroll
            for (int c = 0; c < kChunks; ++c) x[c] = key_nibble(h.w[0], h.w[1], h.w[2], h.w[3], chunk_pos(cp, c));
            for (int32_t g = threadIdx.x; g < G; g += blockDim.x) {
                uint32_t surv = ~0u;
#pragma unroll
                for (int c = 0; c < kChunks; ++c) surv &= fs[static_cast<int64_t>(c * 16 + x[c]) * G + g];
                if (surv) verify_group(surv, rules + rb + static_cast<int64_t>(g) * 32, static_cast<uint32_t>(g) * 32, h,
                                       &best);
            }
            __syncthreads();
            const uint64_t key = best;
            int32_t next = -1;
            uint16_t port = PC_NO_PORT;
            const int state = apply_rule(S, port_off, port_peer, n_ports, ttl, s, key, hops, &next, &port);
            __syncthreads();  // everyone has read `best` before it is reset
            if (state >= 0) {
                if (threadIdx.x == 0) {
                    write_out(out, t, jm, s, port, hops, state);
                    if (visit) visit[t] = vis;
                    if (vsum) vsum[t] = vs;
                }
                break;
            }
            s = next;
            hops += 1;
            jm |= jur_bit(jur, s);
            if (visit) vis |= watch_bits(watch, K, t, s);
            if (vsum) vs |= sum_bit(s);
            if (walk && hops < kWalkSlots && threadIdx.x == 0) walk[static_cast<int64_t>(t) * kWalkSlots + hops] = s;
        }
    }
}

// ---------------------------------------------------------------- deltas
// Summary bits and the bitmap of the changed switches (ids outside [0, S)
// are ignored and raise SWITCH); one workgroup.
__global__ __launch_bounds__(256) void k_delta_mask(const int32_t *__restrict__ changed, int32_t C, int32_t S,
                                                    unsigned long long *__restrict__ mask,
                                                    uint32_t *__restrict__ bitmap, uint32_t *__restrict__ d_err)
{
    __shared__ unsigned long long m;
    if (threadIdx.x == 0) m = 0;
    __syncthreads();
    uint64_t mine = 0;
    bool bad = false;
    for (int32_t i = threadIdx.x; i < C; i += blockDim.x) {
        const int32_t s = changed[i];
        if (s < 0 || s >= S) {
            bad = true;
        } else {
            mine |= sum_bit(s);
            atomicOr(bitmap + (s >> 5), 1u << (s & 31));
        }
    }
    if (mine) atomicOr(&m, static_cast<unsigned long long>(mine));
    if (__ballot(bad) && (threadIdx.x & 63) == 0) atomicOr(d_err, PC_DERR_SWITCH);
    __syncthreads();
    if (threadIdx.x == 0) *mask = m;
}

// The traces to trace again, in a list (one counter update per workgroup
// of 1,024 traces): with walk records, a walk of at most kWalkSlots
// switches (hops + 1 of its record) is selected iff one of them changed;
// otherwise, iff its summary meets the mask.  Also the ingress sweep of the
// SWITCH flag over every trace.
__global__ __launch_bounds__(1024) void k_delta_select(const uint64_t *__restrict__ vsum,
                                                       const int32_t *__restrict__ walk,
                                                       const pc_trace_out *__restrict__ out,
                                                       const uint32_t *__restrict__ bitmap,
                                                       const int32_t *__restrict__ ingress, int32_t T, int32_t S,
                                                       const unsigned long long *__restrict__ mask,
                                                       int32_t *__restrict__ list, uint32_t *__restrict__ count,
                                                       uint32_t *__restrict__ d_err)
{
    __shared__ uint32_t wcount[16], wbase[16];
    const uint64_t m = *mask;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * blockDim.x; base < T;
         base += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t t = base + threadIdx.x;
        const bool in = t < T;
        bool sel = false;
        if (in) {
            const int32_t len = static_cast<int32_t>(out[t].hops) + 1;
            if (walk != nullptr && len <= kWalkSlots) {
                const int32_t *w = walk + t * kWalkSlots;
                for (int j = 0; j < len; ++j) {
                    const int32_t v = w[j];
                    if (v >= 0 && v < S && ((bitmap[v >> 5] >> (v & 31)) & 1u)) sel = true;
                }
            } else {
                sel = (vsum[t] & m) != 0;
            }
        }
        const int32_t s = in ? ingress[t] : 0;
        if (__ballot(in && (s < 0 || s >= S)) && lane == 0) atomicOr(d_err, PC_DERR_SWITCH);
        const uint64_t b = __ballot(sel);
        if (lane == 0) wcount[wave] = static_cast<uint32_t>(__popcll(b));
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t tot = 0;
            for (int w = 0; w < 16; ++w) {
                wbase[w] = tot;
                tot += wcount[w];
            }
            const uint32_t off = tot ? atomicAdd(count, tot) : 0u;
            for (int w = 0; w < 16; ++w) wbase[w] += off;
        }
        __syncthreads();
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(b >> 32),
                                                         __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(b), 0u));
        if (sel) list[wbase[wave] + below] = static_cast<int32_t>(t);
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_delta_gather(const int32_t *__restrict__ list, int32_t n,
                                                      const pc_key *__restrict__ hdr,
                                                      const int32_t *__restrict__ ingress, pc_key *__restrict__ hdr_c,
                                                      int32_t *__restrict__ ing_c)
{
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t t = list[i];
        hdr_c[i] = hdr[t];
        ing_c[i] = ingress[t];
    }
}

__global__ __launch_bounds__(256) void k_delta_scatter(const int32_t *__restrict__ list, int32_t n,
                                                       const pc_trace_out *__restrict__ out_c,
                                                       const uint64_t *__restrict__ vsum_c,
                                                       const int32_t *__restrict__ walk_c,
                                                       pc_trace_out *__restrict__ out, uint64_t *__restrict__ vsum,
                                                       int32_t *__restrict__ walk,
                                                       const uint32_t *__restrict__ count, int32_t *__restrict__ n_out)
{
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        const int32_t t = list[i];
        out[t] = out_c[i];
        vsum[t] = vsum_c[i];
        if (walk)
            for (int j = 0; j < kWalkSlots; ++j)
                walk[static_cast<int64_t>(t) * kWalkSlots + j] = walk_c[static_cast<int64_t>(i) * kWalkSlots + j];
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) *n_out = static_cast<int32_t>(*count);
}

// Cached prepared tables: 1 in *diff when some switch's group count differs
// from the cached one.
__global__ __launch_bounds__(256) void k_tc_compare(const int32_t *__restrict__ gnew, const int32_t *__restrict__ gold,
                                                    int32_t S, uint32_t *__restrict__ diff)
{
    bool d = false;
    for (int32_t s = blockIdx.x * blockDim.x + threadIdx.x; s < S; s += gridDim.x * blockDim.x) d |= gnew[s] != gold[s];
    if (__ballot(d) && (threadIdx.x & 63) == 0) atomicOr(diff, 1u);
}

// Clear the action-error flags of the listed switches (ids outside [0, S) skipped).
__global__ __launch_bounds__(256) void k_tc_clear(const int32_t *__restrict__ changed, int32_t C, int32_t S,
                                                  uint32_t *__restrict__ sw_bad)
{
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < C; i += gridDim.x * blockDim.x) {
        const int32_t s = changed[i];
        if (s >= 0 && s < S) sw_bad[s] = 0;
    }
}

// ACTION when any switch's flag is set.
__global__ __launch_bounds__(256) void k_tc_badsum(const uint32_t *__restrict__ sw_bad, int32_t S,
                                                   uint32_t *__restrict__ d_err)
{
    bool any = false;
    for (int32_t s = blockIdx.x * blockDim.x + threadIdx.x; s < S; s += gridDim.x * blockDim.x) any |= sw_bad[s] != 0;
    if (__ballot(any) && (threadIdx.x & 63) == 0) atomicOr(d_err, PC_DERR_ACTION);
}

unsigned grid_for(int64_t n, int threads)
{
    int64_t b = (n + threads - 1) / threads;
    if (b > 65536) b = 65536;
    return b > 0 ? static_cast<unsigned>(b) : 1u;
}

// Header histogram, then each switch's filter chunks.
int choose_chunks(pc_ctx *ctx, int32_t S, const int32_t *rule_off, int64_t n_rules, const pc_rule *rules,
                  const pc_key *hdr, int32_t T, uint32_t *hh, uint32_t *cpos, hipStream_t stream)
{
    launch_fill_u32(hh, kKeyNibbles * 16, 0, stream);
    if (T > 0)
        PC_TIMED(ctx, "k_tr_hdr_hist", stream,
                 hipLaunchKernelGGL(k_tr_hdr_hist, dim3(64), dim3(256), 0, stream, hdr, T, hh));
    PC_TIMED(ctx, "k_tr_choose", stream,
             hipLaunchKernelGGL(k_tr_choose, dim3(static_cast<unsigned>(S)), dim3(256), 0, stream, S, rule_off,
                                n_rules, rules, hh, cpos));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

}  // namespace

int run_trace(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
              const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
              const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl, const int32_t *watch, int32_t K,
              pc_trace_out *out, uint32_t *visit, uint64_t *vsum, int32_t *walk, hipStream_t stream,
              const TracePrep *pre)
{
    struct Bufs {
        int32_t *gcount, *bcount, *gofs, *bofs, *counts0, *counts1, *boff, *ioff;
        BRec *bucket;
        LRec *live0, *live1;
        int2 *pinfo, *imap;
        uint32_t *filt, *cpos, *hh;
    } B;
    // work items of a level: at most T / kItemCap + S (see the match launch)
    const int32_t icap = static_cast<int32_t>(std::min<int64_t>(static_cast<int64_t>(T) / kItemCap + S + 1, INT32_MAX));
    auto carve = [&](Carver &c) {
        B.cpos = c.take<uint32_t>(S + 1);
        B.hh = c.take<uint32_t>(kKeyNibbles * 16);
        B.gcount = c.take<int32_t>(S + 1);
        B.bcount = c.take<int32_t>(S + 1);
        B.gofs = c.take<int32_t>(S + 1);
        B.bofs = c.take<int32_t>(S + 1);
        B.counts0 = c.take<int32_t>(static_cast<size_t>(S + 1) * kCountPad);
        B.counts1 = c.take<int32_t>(static_cast<size_t>(S + 1) * kCountPad);
        B.boff = c.take<int32_t>(S + 1);
        B.ioff = c.take<int32_t>(S + 1);
        B.live0 = c.take<LRec>(T + 1);
        B.live1 = c.take<LRec>(T + 1);
        B.bucket = c.take<BRec>(T + 1);
        B.pinfo = c.take<int2>(static_cast<size_t>(n_ports) + 1);
        B.imap = c.take<int2>(static_cast<size_t>(icap));
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    // ---- prep: per-switch sizes, offsets, chunk sets, data-error sweep
    // (done by the caller when it passes prepared tables)
    if (pre != nullptr) {
        B.filt = const_cast<uint32_t *>(pre->filt);
        B.gcount = const_cast<int32_t *>(pre->gcount);
        B.gofs = const_cast<int32_t *>(pre->gofs);
        B.cpos = const_cast<uint32_t *>(pre->cpos);
    } else if (S > 0) {
        PC_TIMED(ctx, "k_tr_switch_info", stream, hipLaunchKernelGGL(k_tr_switch_info, dim3(grid_for(S, 256)), dim3(256), 0, stream, S, port_off, n_ports, jur,
                           rule_off, n_rules, B.gcount, B.bcount, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
        launch_scan_i32(B.gcount, S, B.gofs, nullptr, nullptr, stream);
        launch_scan_i32(B.bcount, S, B.bofs, nullptr, nullptr, stream);
        PC_LAUNCH_CHECK(ctx);
        // exact sizes of the chunk-set buffer and of the prep grid (switch
        // ranges may overlap, so no host-side bound from n_rules holds); the
        // host waits for these two counts only, while the port check and
        // the chunk choice, queued behind them, keep the GPU busy
        PC_HIP(ctx, hipMemcpyAsync(ctx->h_small, B.gofs + S, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        PC_HIP(ctx, hipMemcpyAsync(ctx->h_small + 1, B.bofs + S, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        PC_HIP(ctx, hipEventRecord(ctx->lvl_ev[0], stream));
        if (n_ports > 0) {
            PC_TIMED(ctx, "k_tr_port_check", stream, hipLaunchKernelGGL(k_tr_port_check, dim3(grid_for(n_ports, 256)), dim3(256), 0, stream, n_ports,
                               port_peer, S, ctx->d_err));
            PC_LAUNCH_CHECK(ctx);
        }
        rc = choose_chunks(ctx, S, rule_off, n_rules, rules, hdr, T, B.hh, B.cpos, stream);
        if (rc) return rc;
        PC_HIP(ctx, hipEventSynchronize(ctx->lvl_ev[0]));
        const int64_t total_groups = ctx->h_small[0];
        const int64_t prep_blocks = ctx->h_small[1];
        if (total_groups < 0 || prep_blocks < 0)
            return pc_set_error(ctx, PC_EINVAL, "pc_trace_flows: more than 2^31 rule groups");
        rc = pc_ensure_aux(ctx, static_cast<size_t>(total_groups + 1) * kPlaneWords * sizeof(uint32_t));
        if (rc) return rc;
        B.filt = reinterpret_cast<uint32_t *>(ctx->aux);
        if (prep_blocks > 0) {
            PC_TIMED(ctx, "k_tr_prep", stream, hipLaunchKernelGGL(k_tr_prep, dim3(static_cast<unsigned>(prep_blocks)), dim3(kPrepWaves * 64), 0, stream, S,
                               port_off, n_ports, rule_off, rules, B.gcount, B.gofs, B.bofs, B.filt, ctx->d_err,
                               nullptr, nullptr, B.cpos));
            PC_LAUNCH_CHECK(ctx);
        }
    }
    if (T == 0) return PC_OK;
    // the tail walk's workgroup: about two rule groups per lane of a mean
    // table (64-256 threads; 256 when the table sizes are not at hand)
    int walk_threads = 256;
    if (pre == nullptr && S > 0) {
        const int64_t mean_groups = ctx->h_small[0] / S;
        walk_threads = mean_groups <= 128 ? 64 : mean_groups <= 256 ? 128 : 256;
    }
    if (visit && K > 0) {
        PC_TIMED(ctx, "k_tr_watch_check", stream,
                 hipLaunchKernelGGL(k_tr_port_check, dim3(grid_for(static_cast<int64_t>(T) * K, 256)), dim3(256), 0,
                                    stream, static_cast<int64_t>(T) * K, watch, S, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (!visit) K = 0;
    if (n_ports > 0) {
        PC_TIMED(ctx, "k_tr_port_info", stream,
                 hipLaunchKernelGGL(k_tr_port_info, dim3(static_cast<unsigned>(std::min<int64_t>((n_ports + 255) / 256, 4096))),
                                    dim3(256), 0, stream, n_ports, port_peer, S, jur, B.pinfo));
        PC_LAUNCH_CHECK(ctx);
    }

    // ---- level-synchronous walk
    int32_t *d_n = ctx->d_small;  // [0], [1]: live counts of the two live lists ([4], [5]: the reach kernels')
    launch_fill_u32(reinterpret_cast<uint32_t *>(d_n), 2, 0, stream);
    if (S > 0) {
        launch_fill_u32(reinterpret_cast<uint32_t *>(B.counts0), static_cast<size_t>(S + 1) * kCountPad, 0, stream);
        launch_fill_u32(reinterpret_cast<uint32_t *>(B.counts1), static_cast<size_t>(S + 1) * kCountPad, 0, stream);
    }
    {
        const dim3 ig(static_cast<unsigned>((static_cast<int64_t>(T) + kInitPer - 1) / kInitPer));
        if (S <= kInitLdsS)
            PC_TIMED(ctx, "k_tr_init", stream,
                     hipLaunchKernelGGL(k_tr_init<true>, ig, dim3(kInitThreads), static_cast<size_t>(S) * 4, stream, S,
                                        jur, ingress, hdr, T, B.live0, d_n, B.counts0, out, watch, K, visit, vsum,
                                        walk, ctx->d_err));
        else
            PC_TIMED(ctx, "k_tr_init", stream,
                     hipLaunchKernelGGL(k_tr_init<false>, ig, dim3(kInitThreads), 0, stream, S, jur, ingress, hdr, T,
                                        B.live0, d_n, B.counts0, out, watch, K, visit, vsum, walk, ctx->d_err));
    }
    PC_LAUNCH_CHECK(ctx);
    LRec *live_cur = B.live0, *live_nxt = B.live1;
    int32_t *cnt_cur = B.counts0, *cnt_nxt = B.counts1;
    int32_t *n_cur = d_n, *n_nxt = d_n + 1;
    // Levels with few traces in flight are cheaper as independent walks than
    // as bucketed passes (tunable with PC_TRACE_WALK_MAX, 0 = never walk).
    int64_t walk_max = 8192;
    if (const char *env = getenv("PC_TRACE_WALK_MAX")) walk_max = atoll(env);
    // The host does not wait for a level before queueing the next one: live
    // counts only shrink, so level L is launched with the latest count the
    // host has (exact for level 0, else the count entering level L - 1) as
    // the bound for its grids, and the kernels read the exact count on the
    // device.  The count entering level L is copied back after level L - 1
    // and waited for (an event one level behind) while level L runs.
    int32_t *h_cnt = ctx->h_small + 8;  // two pinned slots, by level parity
    int32_t *d_len = ctx->d_small + 6;  // two slots, by level parity: each level's lookups (its live list's length)
    // An upper bound on the count entering the next level (T for level 0:
    // the host does not wait for the initial count); from level 2 on, also
    // the exact length of the live list the previous level wrote (every
    // lookup of a level leaves an entry, the traces that ended included).
    int64_t known = T;
    for (int level = 0;; ++level) {
        if (level > ttl + 2)
            return pc_set_error(ctx, PC_EDEVICE, "pc_trace_flows: level loop exceeded ttl+2 levels");
        if (known == 0) break;
        // the live list this level reads: from k_tr_init (as many entries as
        // traces in flight) or from the previous level's match
        const int32_t *len_cur = level == 0 ? n_cur : d_len + ((level - 1) & 1);
        if (known <= walk_max) {
            const unsigned wb = static_cast<unsigned>(known < 8192 ? known : 8192);
            PC_TIMED(ctx, "k_tr_walk", stream,
                     hipLaunchKernelGGL(k_tr_walk, dim3(wb), dim3(walk_threads), 0, stream, S, port_off, port_peer, n_ports, jur,
                                        rule_off, rules, B.gcount, B.gofs, B.filt, ttl, live_cur, len_cur, level,
                                        out, watch, K, visit, vsum, walk, B.cpos));
            PC_LAUNCH_CHECK(ctx);
            break;
        }
        const int32_t nlive = static_cast<int32_t>(known);
        PC_TIMED(ctx, "k_tr_plan", stream,
                 hipLaunchKernelGGL(k_tr_plan, dim3(1), dim3(1024), 0, stream, cnt_cur, S, B.boff, B.ioff,
                                    B.gcount, d_len + (level & 1), n_nxt));
        PC_TIMED(ctx, "k_tr_scatter", stream,
                 hipLaunchKernelGGL(k_tr_scatter, dim3(grid_for(nlive, 256)), dim3(256), 0, stream, live_cur, len_cur,
                                    T, S, B.boff, B.bucket, B.ioff, B.imap, icap));
        const Level lv{S,        T,     port_off, port_peer, B.pinfo, n_ports, jur,   ttl,  level,
                       live_nxt, n_nxt, cnt_nxt,  out,       watch,   K,       visit, vsum, walk};
        // at most nlive / kItemCap + S items: a switch of n lookups takes ceil(n / cap) items with cap >= kItemCap
        const int64_t max_items = std::min<int64_t>(static_cast<int64_t>(nlive) / kItemCap + S, nlive);
        PC_TIMED(ctx, "k_tr_match", stream,
                 hipLaunchKernelGGL(k_tr_match, dim3(static_cast<unsigned>(8 * ((max_items + 7) / 8))),
                                    dim3(kMatchThreads), 0, stream, S, rule_off, rules, B.gcount, B.gofs, B.filt,
                                    B.boff, B.ioff, B.imap, B.bucket, B.cpos, lv));
        PC_LAUNCH_CHECK(ctx);
        // the count leaving this level
        const int slot = (level + 1) & 1;
        PC_HIP(ctx, hipMemcpyAsync(h_cnt + slot, n_nxt, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        PC_HIP(ctx, hipEventRecord(ctx->lvl_ev[slot], stream));
        if (level == 0) {
            known = nlive;  // the bound for level 1; its exact count is learned after level 0 completes
        } else {
            // the count entering this level (left by the previous level): its
            // copy completed before this level started
            PC_HIP(ctx, hipEventSynchronize(ctx->lvl_ev[level & 1]));
            known = h_cnt[level & 1];
        }
        std::swap(live_cur, live_nxt);
        int32_t *tmp;
        tmp = cnt_cur; cnt_cur = cnt_nxt; cnt_nxt = tmp;
        tmp = n_cur; n_cur = n_nxt; n_nxt = tmp;
    }
    return PC_OK;
}

namespace {

// Per-switch arrays of the cached prepared tables in ctx->tc_meta.
struct TcMeta {
    int32_t *gcount, *bcount, *gofs, *bofs;
    uint32_t *sw_bad, *cpos, *hh;
};

TcMeta tc_meta(pc_ctx *ctx, int32_t S)
{
    Carver c{ctx->tc_meta, 0};
    TcMeta m;
    m.gcount = c.take<int32_t>(static_cast<size_t>(S) + 1);
    m.bcount = c.take<int32_t>(static_cast<size_t>(S) + 1);
    m.gofs = c.take<int32_t>(static_cast<size_t>(S) + 1);
    m.bofs = c.take<int32_t>(static_cast<size_t>(S) + 1);
    m.sw_bad = c.take<uint32_t>(static_cast<size_t>(S) + 1);
    m.cpos = c.take<uint32_t>(static_cast<size_t>(S) + 1);
    m.hh = c.take<uint32_t>(kKeyNibbles * 16);
    return m;
}

size_t tc_meta_bytes(int32_t S) { return 7 * (256 + (static_cast<size_t>(S) + 1) * 4) + kKeyNibbles * 16 * 4; }

// Prepare every switch's tables into the context's cache (and sweep them
// for data errors); the cache then describes these tables.
int tc_prepare_all(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                   const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
                   const pc_key *hdr, int32_t T, hipStream_t stream)
{
    ctx->tc_S = -1;
    int rc = pc_ensure_tc_meta(ctx, tc_meta_bytes(S));
    if (rc) return rc;
    const TcMeta m = tc_meta(ctx, S);
    int64_t groups = 0, blocks = 0;
    if (S > 0) {
        PC_TIMED(ctx, "k_tr_switch_info", stream,
                 hipLaunchKernelGGL(k_tr_switch_info, dim3(grid_for(S, 256)), dim3(256), 0, stream, S, port_off,
                                    n_ports, jur, rule_off, n_rules, m.gcount, m.bcount, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
        launch_scan_i32(m.gcount, S, m.gofs, nullptr, nullptr, stream);
        launch_scan_i32(m.bcount, S, m.bofs, nullptr, nullptr, stream);
        PC_LAUNCH_CHECK(ctx);
        PC_HIP(ctx, hipMemcpyAsync(ctx->h_small, m.gofs + S, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        PC_HIP(ctx, hipMemcpyAsync(ctx->h_small + 1, m.bofs + S, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        PC_HIP(ctx, hipStreamSynchronize(stream));
        groups = ctx->h_small[0];
        blocks = ctx->h_small[1];
        if (groups < 0 || blocks < 0)
            return pc_set_error(ctx, PC_EINVAL, "pc_trace_flows_delta: more than 2^31 rule groups");
    }
    rc = pc_ensure_tc_filt(ctx, static_cast<size_t>(groups + 1) * kPlaneWords * sizeof(uint32_t));
    if (rc) return rc;
    if (S > 0) {
        if (n_ports > 0) {
            PC_TIMED(ctx, "k_tr_port_check", stream,
                     hipLaunchKernelGGL(k_tr_port_check, dim3(grid_for(n_ports, 256)), dim3(256), 0, stream, n_ports,
                                        port_peer, S, ctx->d_err));
            PC_LAUNCH_CHECK(ctx);
        }
        launch_fill_u32(m.sw_bad, static_cast<size_t>(S), 0, stream);
        rc = choose_chunks(ctx, S, rule_off, n_rules, rules, hdr, T, m.hh, m.cpos, stream);
        if (rc) return rc;
        if (blocks > 0) {
            PC_TIMED(ctx, "k_tr_prep", stream,
                     hipLaunchKernelGGL(k_tr_prep, dim3(static_cast<unsigned>(blocks)), dim3(kPrepWaves * 64), 0,
                                        stream, S, port_off, n_ports, rule_off, rules, m.gcount, m.gofs, m.bofs,
                                        reinterpret_cast<uint32_t *>(ctx->tc_filt), ctx->d_err, nullptr, m.sw_bad,
                                        m.cpos));
            PC_LAUNCH_CHECK(ctx);
        }
    }
    ctx->tc_S = S;
    ctx->tc_groups = groups;
    ctx->tc_blocks = blocks;
    return PC_OK;
}

}  // namespace

int run_trace_delta(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                    const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
                    const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl, const int32_t *changed,
                    int32_t C, pc_trace_out *out, uint64_t *vsum, int32_t *walk, int32_t *n_retraced,
                    hipStream_t stream)
{
    if (C < 0) {  // every trace, from scratch; the prepared tables are kept for later deltas
        launch_fill_u32(reinterpret_cast<uint32_t *>(n_retraced), 1, static_cast<uint32_t>(T), stream);
        int rc = tc_prepare_all(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, T, stream);
        if (rc) return rc;
        if (T == 0) return PC_OK;
        const TcMeta m = tc_meta(ctx, S);
        const TracePrep pre{reinterpret_cast<const uint32_t *>(ctx->tc_filt), m.gcount, m.gofs, m.cpos};
        return run_trace(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, ingress, T, ttl,
                         nullptr, 0, out, nullptr, vsum, walk, stream, &pre);
    }
    // compacted traces live in their own buffer: run_trace carves the arena
    const size_t Tn = static_cast<size_t>(T) + 1;
    const size_t words = (static_cast<size_t>(S) + 31) / 32 + 1;
    const size_t need = 256 * 14 + words * 4 + 2 * (static_cast<size_t>(S) + 1) * 4 +
                        Tn * (sizeof(int32_t) * 2 + sizeof(pc_key) + sizeof(pc_trace_out) + 8 + 4 * kWalkSlots);
    int rc = pc_ensure_delta(ctx, need);
    if (rc) return rc;
    Carver cv{ctx->delta, 0};
    unsigned long long *mask = cv.take<unsigned long long>(1);
    uint32_t *count = cv.take<uint32_t>(2);  // [0] selected traces, [1] a group count differs from the cache
    int32_t *list = cv.take<int32_t>(Tn);
    pc_key *hdr_c = cv.take<pc_key>(Tn);
    int32_t *ing_c = cv.take<int32_t>(Tn);
    pc_trace_out *out_c = cv.take<pc_trace_out>(Tn);
    uint64_t *vsum_c = cv.take<uint64_t>(Tn);
    int32_t *walk_c = cv.take<int32_t>(Tn * kWalkSlots);
    uint32_t *bitmap = cv.take<uint32_t>(words);
    int32_t *gnew = cv.take<int32_t>(static_cast<size_t>(S) + 1);
    int32_t *bnew = cv.take<int32_t>(static_cast<size_t>(S) + 1);
    launch_fill_u32(count, 2, 0, stream);
    launch_fill_u32(bitmap, words, 0, stream);
    PC_TIMED(ctx, "k_delta_mask", stream,
             hipLaunchKernelGGL(k_delta_mask, dim3(1), dim3(256), 0, stream, changed, C, S, mask, bitmap,
                                ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    if (T > 0) {
        PC_TIMED(ctx, "k_delta_select", stream,
                 hipLaunchKernelGGL(k_delta_select, dim3(grid_for(T, 1024)), dim3(1024), 0, stream, vsum, walk, out,
                                    bitmap, ingress, T, S, mask, list, count, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    // with reuse declared (pc_trace_keep_tables) the cache holds the previous
    // tables when its switch count matches; it serves the new ones when no
    // switch's group count changed.  Without it every call prepares anew.
    const bool cached = ctx->tc_keep && ctx->tc_S == S && S > 0;
    if (cached) {
        const TcMeta m = tc_meta(ctx, S);
        PC_TIMED(ctx, "k_tr_switch_info", stream,
                 hipLaunchKernelGGL(k_tr_switch_info, dim3(grid_for(S, 256)), dim3(256), 0, stream, S, port_off,
                                    n_ports, jur, rule_off, n_rules, gnew, bnew, ctx->d_err));
        PC_TIMED(ctx, "k_tc_compare", stream,
                 hipLaunchKernelGGL(k_tc_compare, dim3(grid_for(S, 256)), dim3(256), 0, stream, gnew, m.gcount, S,
                                    count + 1));
        PC_LAUNCH_CHECK(ctx);
    }
    PC_HIP(ctx, hipMemcpyAsync(ctx->h_small, count, 2 * sizeof(uint32_t), hipMemcpyDeviceToHost, stream));
    PC_HIP(ctx, hipStreamSynchronize(stream));
    const int32_t n = ctx->h_small[0];
    if (cached && ctx->h_small[1] == 0) {
        // re-prepare only the changed switches, then the ACTION flag over all
        const TcMeta m = tc_meta(ctx, S);
        if (n_ports > 0) {
            PC_TIMED(ctx, "k_tr_port_check", stream,
                     hipLaunchKernelGGL(k_tr_port_check, dim3(grid_for(n_ports, 256)), dim3(256), 0, stream, n_ports,
                                        port_peer, S, ctx->d_err));
        }
        if (C > 0) {
            PC_TIMED(ctx, "k_tc_clear", stream,
                     hipLaunchKernelGGL(k_tc_clear, dim3(grid_for(C, 256)), dim3(256), 0, stream, changed, C, S,
                                        m.sw_bad));
        }
        if (ctx->tc_blocks > 0 && C > 0) {
            // the changed switches keep their filter chunks (any choice is exact)
            PC_TIMED(ctx, "k_tr_prep", stream,
                     hipLaunchKernelGGL(k_tr_prep, dim3(static_cast<unsigned>(ctx->tc_blocks)), dim3(kPrepWaves * 64),
                                        0, stream, S, port_off, n_ports, rule_off, rules, m.gcount, m.gofs, m.bofs,
                                        reinterpret_cast<uint32_t *>(ctx->tc_filt), ctx->d_err, bitmap, m.sw_bad,
                                        m.cpos));
        }
        PC_TIMED(ctx, "k_tc_badsum", stream,
                 hipLaunchKernelGGL(k_tc_badsum, dim3(grid_for(S, 256)), dim3(256), 0, stream, m.sw_bad, S,
                                    ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    } else {
        rc = tc_prepare_all(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, T, stream);
        if (rc) return rc;
    }
    if (n > 0) {
        PC_TIMED(ctx, "k_delta_gather", stream,
                 hipLaunchKernelGGL(k_delta_gather, dim3(grid_for(n, 256)), dim3(256), 0, stream, list, n, hdr,
                                    ingress, hdr_c, ing_c));
        PC_LAUNCH_CHECK(ctx);
        const TcMeta m = tc_meta(ctx, S);
        const TracePrep pre{reinterpret_cast<const uint32_t *>(ctx->tc_filt), m.gcount, m.gofs, m.cpos};
        rc = run_trace(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr_c, ing_c, n, ttl,
                       nullptr, 0, out_c, nullptr, vsum_c, walk ? walk_c : nullptr, stream, &pre);
        if (rc) return rc;
    }
    PC_TIMED(ctx, "k_delta_scatter", stream,
             hipLaunchKernelGGL(k_delta_scatter, dim3(grid_for(n > 0 ? n : 1, 256)), dim3(256), 0, stream, list, n,
                                out_c, vsum_c, walk_c, out, vsum, walk, count, n_retraced));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

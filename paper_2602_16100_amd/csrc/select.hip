// A1 -- placement constraints: node-selector evaluation for every selector
// row x node, emitting a feasible-node bitset and a popcount per row.
//
// The operators are Kubernetes node-affinity's (In / NotIn / Exists over a
// label), which is how the paper compiles a placement constraint such as
// "region=EU is among the labels of the node the pod is placed on" (Formal
// Model and Satisfaction, example; Service Placement Module).
//
// Design (gfx950):
//   1. presence  : which values of each label occur at all.
//   2. label scan: plane numbering -- one plane per present (label, value).
//   3. planes    : one 64-bit node set per (plane, 64-node word), built with
//                  a ballot per present value; row-major, Wp words a plane.
//   4. compile   : one thread per row turns its predicates into a clause
//                  program over plane ids (In S = OR of S's planes or NOT OR
//                  of the rest, whichever is shorter; NotIn the reverse;
//                  Exists = NOT the absent-value plane), validates it, and
//                  writes a 64-byte row record holding programs of up to 15
//                  entries inline.
//   5. eval      : one row at a time per wavefront over a tile of 128 words
//                  (two per lane, 16-byte loads and stores).  The row's
//                  record arrives through scalar loads, so its plane loads
//                  (L2 hits: a tile of every plane is P KiB) all go out
//                  together with scalar offsets, followed by one output
//                  store.  Per-lane popcounts are collected as bytes in LDS
//                  and summed once per 64 rows; a last pass sums the tiles.
#include <algorithm>

#include "pc_internal.h"

namespace {

constexpr int kEvalThreads = 256;  // 4 wavefronts, one row at a time each
constexpr int kWpl = 2;            // 64-bit words per lane
constexpr int kTileW = 64 * kWpl;  // words per tile
constexpr int kRecWords = 16;      // row record: header + 15 inline entries
constexpr int kInline = kRecWords - 1;
constexpr int kGroup = 8;          // plane loads in flight together

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
    uint32_t m[8] = {0, 0, 0, 0, 0, 0, 0, 0};  // this thread's 256-bit value set, in registers
    if (l < L) {
        for (int64_t n = n0 + sub; n < n1; n += 4) {
            const uint32_t x = labels[n * L + l];
            const uint32_t word = x >> 5, bit = 1u << (x & 31);
#pragma unroll
            for (int k = 0; k < 8; ++k) m[k] |= word == static_cast<uint32_t>(k) ? bit : 0u;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (m[k]) atomicOr(&tab[lt * 8 + k], m[k]);
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
                                                         uint32_t *__restrict__ wbase, int32_t *__restrict__ d_P)
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
    if (tid == 0) *d_P = static_cast<int32_t>(carry_s);
}

// One wavefront per (64-node word w, label l): a ballot per present value.
// Word w of plane p lives at planes[p * Wp + w].
__global__ __launch_bounds__(256) void k_sel_planes(const uint8_t *__restrict__ labels, int32_t N, int32_t L,
                                                    const uint64_t *__restrict__ present,
                                                    const uint32_t *__restrict__ wbase, uint64_t *__restrict__ planes,
                                                    int64_t Wp)
{
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t w = blockIdx.x;
    const int32_t l = blockIdx.y * 4 + wave;
    if (l >= L) return;
    uint64_t *col = planes + w;
    const int64_t n = static_cast<int64_t>(w) * 64 + lane;
    const uint32_t x = n < N ? labels[n * L + l] : 0x100u;  // 0x100 equals no value
    for (int k = 0; k < 4; ++k) {
        uint64_t m = uniform_u64(present[static_cast<int64_t>(l) * 4 + k]);
        uint32_t pid = __builtin_amdgcn_readfirstlane(wbase[static_cast<int64_t>(l) * 4 + k]);
        while (m) {
            const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
            const uint64_t word = __ballot(x == v);
            if (lane == 0) col[static_cast<int64_t>(pid) * Wp] = word;
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
// Row record header (word 0); words 1..15 hold an inline program.
constexpr int32_t kRowFalse = -1;     // some clause admits no node (or a malformed predicate)
constexpr int32_t kRowIndirect = -2;  // program of more than 15 entries at prog[4 * word1], word2 entries
constexpr int32_t kRowLong = -3;      // program longer than 4 entries per predicate: decoded on the fly

__device__ __forceinline__ uint32_t plane_id(const uint64_t *pres, const uint32_t *wb, uint32_t v)
{
    const uint32_t k = v >> 6;
    return wb[k] + __popcll(pres[k] & ((1ull << (v & 63)) - 1));
}

// The value set a predicate ORs over, and whether the OR is negated.  Each
// label value of a node lies in exactly one present plane, so In S = OR(S)
// = NOT OR(present \ S) and NotIn S = NOT OR(S) = OR(present \ S): the
// shorter form is taken.  Exists = NOT OR(plane of the absent value), an
// empty OR when every node carries the label.
__device__ __forceinline__ uint32_t pred_clause(const pc_pred &q, const uint64_t *pres, uint64_t sel[4], bool &neg)
{
    if (q.op == PC_OP_EXISTS) {
        sel[0] = sel[1] = sel[2] = 0;
        sel[3] = pres[3] & (1ull << 63);
        neg = true;
        return static_cast<uint32_t>(sel[3] >> 63);
    }
    uint64_t in[4], out[4];
    uint32_t ms = 0, mc = 0;
    for (int k = 0; k < 4; ++k) {
        in[k] = q.vals[k] & pres[k];
        out[k] = pres[k] & ~q.vals[k];
        ms += __popcll(in[k]);
        mc += __popcll(out[k]);
    }
    const bool use_in = ms <= mc;
    for (int k = 0; k < 4; ++k) sel[k] = use_in ? in[k] : out[k];
    neg = (q.op == PC_OP_IN) ? !use_in : use_in;
    return use_in ? ms : mc;
}

// One thread per row, two passes over its predicates: validate and size
// the program, then emit it -- inline in the row record when it has at most
// 15 entries, else at prog[4 * pred_off[i] ...] (at most 4 entries per
// predicate; longer programs are decoded at evaluation time).
__global__ __launch_bounds__(256) void k_sel_compile(const int32_t *__restrict__ pred_off,
                                                     const pc_pred *__restrict__ preds, int64_t n_preds, int32_t I,
                                                     int32_t L, const uint64_t *__restrict__ present,
                                                     const uint32_t *__restrict__ wbase, uint32_t zero_pid,
                                                     uint32_t *__restrict__ prog, uint32_t *__restrict__ rec,
                                                     uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < I; i += gridDim.x * blockDim.x) {
        uint32_t *rr = rec + static_cast<int64_t>(i) * kRecWords;
        const int64_t b = pred_off[i], e = pred_off[i + 1];
        if (!pc_range_ok(b, e, n_preds)) {
            errs |= PC_DERR_OFFSETS;
            rr[0] = static_cast<uint32_t>(kRowFalse);
            continue;
        }
        bool empty = false;
        int64_t n = 0;
        for (int64_t p = b; p < e; ++p) {
            const pc_pred q = preds[p];
            if (!pred_valid(q.label, q.op, q.rsv0, q.rsv1, q.vals[3], L)) {
                errs |= PC_DERR_PRED;
                empty = true;
                continue;
            }
            uint64_t sel[4];
            bool neg;
            const uint32_t cnt = pred_clause(q, present + static_cast<int64_t>(q.label) * 4, sel, neg);
            if (cnt == 0 && !neg) empty = true;  // empty OR: no node (a negated empty OR is every node)
            n += cnt;
        }
        if (empty) {
            rr[0] = static_cast<uint32_t>(kRowFalse);
            continue;
        }
        const bool inl = n <= kInline;
        if (!inl && n > 4 * (e - b)) {
            rr[0] = static_cast<uint32_t>(kRowLong);
            continue;
        }
        uint32_t *out = inl ? rr + 1 : prog + 4 * b;
        int64_t k_out = 0;
        for (int64_t p = b; p < e; ++p) {
            const pc_pred q = preds[p];
            const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
            const uint32_t *wb = wbase + static_cast<int64_t>(q.label) * 4;
            uint64_t sel[4];
            bool neg;
            uint32_t cnt = pred_clause(q, pres, sel, neg);
            for (int k = 0; k < 4; ++k) {
                uint64_t m = sel[k];
                while (m) {
                    const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                    m &= m - 1;
                    uint32_t ent = plane_id(pres, wb, v);
                    if (--cnt == 0) ent |= kLast | (neg ? kNeg : 0u);
                    out[k_out++] = ent;
                }
            }
        }
        if (inl) {
            // pad to a whole group (8, or all 15 slots) with the all-zero
            // plane, which changes no clause: evaluation then needs no
            // per-entry bound checks
            const int64_t padded = n == 0 ? 0 : (n <= kGroup ? kGroup : kInline);
            for (int64_t k = n; k < padded; ++k) rr[1 + k] = zero_pid;
            rr[0] = static_cast<uint32_t>(n);
        } else {
            rr[0] = static_cast<uint32_t>(kRowIndirect);
            rr[1] = static_cast<uint32_t>(b);
            rr[2] = static_cast<uint32_t>(n);
        }
    }
    if (errs) atomicOr(d_err, errs);
}

struct Words {
    uint64_t a, b;
};
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ Words load_words(const uint64_t *p)
{
    const ulonglong2 v = *reinterpret_cast<const ulonglong2 *>(p);
    return {v.x, v.y};
}

// Fold one program entry's plane words into the running clause (c) and,
// at the end of a clause, into the row's conjunction (a).
__device__ __forceinline__ void fold(uint32_t ent, const Words &v, Words &c, Words &a)
{
    c.a |= v.a;
    c.b |= v.b;
    if (ent & kLast) {
        if (ent & kNeg) {
            a.a &= ~c.a;
            a.b &= ~c.b;
        } else {
            a.a &= c.a;
            a.b &= c.b;
        }
        c.a = c.b = 0;
    }
}

// This lane's two words of plane `pid`.  The buffer form (planes within
// 4 GiB) takes the plane offset as a scalar operand: one scalar multiply
// per load and no vector address arithmetic.
template <bool kBuf>
struct Planes {
    __amdgpu_buffer_rsrc_t rsrc;
    uint32_t lane_off;  // bytes: this lane's first word within a plane row
    uint32_t rowbytes;  // bytes per plane row
    const uint64_t *pcol;
    int64_t Wp;

    __device__ __forceinline__ Words operator()(uint32_t pid) const
    {
        if constexpr (kBuf) {
            const u32x4 v = __builtin_bit_cast(
                u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, lane_off, pid * rowbytes, 0));
            return {static_cast<uint64_t>(v.x) | static_cast<uint64_t>(v.y) << 32,
                    static_cast<uint64_t>(v.z) | static_cast<uint64_t>(v.w) << 32};
        } else {
            return load_words(pcol + static_cast<int64_t>(pid) * Wp);
        }
    }
};

// Rows whose program did not fit its slot: decode the predicates on the
// scalar unit.
template <bool kBuf>
__device__ Words eval_row_decoded(const pc_pred *__restrict__ preds, int64_t b, int64_t e,
                                  const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
                                  const Planes<kBuf> &pl)
{
    Words a{~0ull, ~0ull};
    for (int64_t p = b; p < e; ++p) {
        const pc_pred *q = preds + p;
        const uint32_t label = q->label, op = q->op;
        const uint64_t *pres = present + static_cast<int64_t>(label) * 4;
        const uint32_t *wb = wbase + static_cast<int64_t>(label) * 4;
        if (op == PC_OP_EXISTS) {
            if (pres[3] >> 63) {
                const Words v = pl(plane_id(pres, wb, 255));
                a.a &= ~v.a;
                a.b &= ~v.b;
            }
            continue;
        }
        Words c{0, 0};
        for (int k = 0; k < 4; ++k) {
            uint64_t m = q->vals[k] & pres[k];
            while (m) {
                const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                m &= m - 1;
                const Words x = pl(plane_id(pres, wb, v));
                c.a |= x.a;
                c.b |= x.b;
            }
        }
        if (op == PC_OP_IN) {
            a.a &= c.a;
            a.b &= c.b;
        } else {
            a.a &= ~c.a;
            a.b &= ~c.b;
        }
    }
    return a;
}

// Work item (tile, chunk): the wavefronts of a workgroup take turns on
// batches of 64 consecutive rows of the chunk; lane l covers words
// tile * 128 + 2l and + 1.  A row's record is read with scalar loads (the
// next row's is requested while the current row's planes load), so the
// plane loads of a row are all in flight together.  Each lane leaves its
// popcount of row i as byte (i, lane) of an LDS table; at the end of a
// batch lane i sums row i's 64 bytes with dot4 and stores
// part[tile * I + r].  Lanes past the last word load in-bounds words and
// mask them.
template <bool kBuf>
__global__ __launch_bounds__(kEvalThreads) void k_sel_eval(
    const uint32_t *__restrict__ rec, const uint32_t *__restrict__ prog, const int32_t *__restrict__ pred_off,
    const pc_pred *__restrict__ preds, const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
    const uint64_t *__restrict__ planes, int64_t plane_bytes, int64_t Wp, int32_t I, int32_t W, int32_t N,
    uint64_t *__restrict__ feasible, uint32_t *__restrict__ part, int32_t ntiles, int32_t nchunks, int32_t rpc)
{
    constexpr int kCntStride = 68;  // bytes per row of the count table (17 dwords: conflict-free column reads)
    __shared__ uint32_t cnt_lds[kEvalThreads / 64][64 * kCntStride / 4];
    const int64_t total = static_cast<int64_t>(ntiles) * nchunks;
    const int64_t item = pc_xcd_item(total);
    if (item >= total) return;
    const int32_t tile = static_cast<int32_t>(item / nchunks);
    const int32_t chunk = static_cast<int32_t>(item % nchunks);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t w0 = tile * kTileW + lane * kWpl;
    const bool ok0 = w0 < W, ok1 = w0 + 1 < W;
    const uint64_t last = (N & 63) ? (1ull << (N & 63)) - 1 : ~0ull;
    const uint64_t m0 = ok0 ? (w0 == W - 1 ? last : ~0ull) : 0ull;
    const uint64_t m1 = ok1 ? (w0 + 1 == W - 1 ? last : ~0ull) : 0ull;
    const int32_t wl = ok0 ? w0 : 0;  // in-bounds column for lanes past the last word
    Planes<kBuf> pl;
    if constexpr (kBuf)
        pl.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(planes), static_cast<short>(0),
                                                    static_cast<int>(plane_bytes), 0x00020000);
    pl.lane_off = static_cast<uint32_t>(wl) * 8u;
    pl.rowbytes = static_cast<uint32_t>(Wp * 8);
    pl.pcol = planes + wl;
    pl.Wp = Wp;
    const bool even = (W & 1) == 0;
    uint8_t *cb = reinterpret_cast<uint8_t *>(cnt_lds[wave]);
    uint32_t *prt = part + static_cast<int64_t>(tile) * I;
    const int32_t r0 = chunk * rpc;
    const int32_t r1 = min(I, r0 + rpc);
    // one row: its record R (uniform, in SGPRs) -> bitset store and count byte
    auto row = [&](int32_t r, int32_t i, const uint32_t (&R)[kRecWords]) {
        const int32_t hdr = static_cast<int32_t>(R[0]);
        Words a{~0ull, ~0ull};
        if (hdr == kRowFalse) {
            a = Words{0, 0};
        } else if (hdr > 0) {
            // inline program, padded with the zero plane to 8 or 15 entries
            Words c{0, 0};
            {
                Words V[kGroup];
#pragma unroll
                for (int k = 0; k < kGroup; ++k) V[k] = pl(R[1 + k] & kPidMask);
#pragma unroll
                for (int k = 0; k < kGroup; ++k) fold(R[1 + k], V[k], c, a);
            }
            if (hdr > kGroup) {
                Words V[kInline - kGroup];
#pragma unroll
                for (int k = 0; k < kInline - kGroup; ++k) V[k] = pl(R[1 + kGroup + k] & kPidMask);
#pragma unroll
                for (int k = 0; k < kInline - kGroup; ++k) fold(R[1 + kGroup + k], V[k], c, a);
            }
        } else if (hdr == kRowIndirect) {
            const uint32_t *pr = prog + 4 * static_cast<int64_t>(R[1]);
            const int32_t len = static_cast<int32_t>(R[2]);
            Words c{0, 0};
            for (int32_t e0 = 0; e0 < len; e0 += kGroup) {
                uint32_t E[kGroup];
                Words V[kGroup];
#pragma unroll
                for (int k = 0; k < kGroup; ++k) E[k] = (e0 + k < len) ? pr[e0 + k] : 0u;
#pragma unroll
                for (int k = 0; k < kGroup; ++k)
                    if (e0 + k < len) V[k] = pl(E[k] & kPidMask);
#pragma unroll
                for (int k = 0; k < kGroup; ++k)
                    if (e0 + k < len) fold(E[k], V[k], c, a);
            }
        } else if (hdr == kRowLong) {
            a = eval_row_decoded<kBuf>(preds, pred_off[r], pred_off[r + 1], present, wbase, pl);
        }
        a.a &= m0;
        a.b &= m1;
        uint64_t *dst = feasible + static_cast<int64_t>(r) * W + w0;
        if (even) {
            if (ok0) __builtin_nontemporal_store(u64x2{a.a, a.b}, reinterpret_cast<u64x2 *>(dst));
        } else {
            if (ok0) __builtin_nontemporal_store(a.a, dst);
            if (ok1) __builtin_nontemporal_store(a.b, dst + 1);
        }
        cb[i * kCntStride + lane] = static_cast<uint8_t>(__popcll(a.a) + __popcll(a.b));
    };
    auto load_rec = [&](int32_t r, uint32_t (&R)[kRecWords]) {
        const uint32_t *rp = rec + static_cast<int64_t>(r) * kRecWords;
#pragma unroll
        for (int k = 0; k < kRecWords; ++k) R[k] = rp[k];
    };
    for (int32_t bat = r0 + wave * 64; bat < r1; bat += kEvalThreads) {
        const int32_t nb = min(64, r1 - bat);
        // two record buffers: the next row's record loads while this row's
        // planes load (the last row reloads its own record)
        uint32_t RA[kRecWords], RB[kRecWords];
        load_rec(bat, RA);
        for (int32_t i = 0; i < nb; i += 2) {
            load_rec(bat + min(i + 1, nb - 1), RB);
            row(bat + i, i, RA);
            if (i + 1 < nb) {
                load_rec(bat + min(i + 2, nb - 1), RA);
                row(bat + i + 1, i + 1, RB);
            }
        }
        // the count table was written by every lane of this wavefront
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (lane < nb) {
            const uint32_t *row = cnt_lds[wave] + lane * (kCntStride / 4);
            uint32_t sum = 0;
#pragma unroll
            for (int k = 0; k < 16; ++k) sum = __builtin_amdgcn_udot4(row[k], 0x01010101u, sum, false);
            prt[bat + lane] = sum;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// popcnt[r] = sum over tiles of part[t * I + r].
__global__ __launch_bounds__(256) void k_sel_popsum(const uint32_t *__restrict__ part, int32_t I, int32_t ntiles,
                                                    uint32_t *__restrict__ popcnt)
{
    const int32_t r = blockIdx.x * 256 + threadIdx.x;
    if (r >= I) return;
    uint32_t s = 0;
    for (int32_t t = 0; t < ntiles; ++t) s += part[static_cast<int64_t>(t) * I + r];
    popcnt[r] = s;
}

}  // namespace

int run_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                  const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                  hipStream_t stream)
{
    const int64_t W = (static_cast<int64_t>(N) + 63) / 64;
    const int64_t Wp = (W + 1) / 2 * 2;  // even: 16-byte aligned plane rows
    const int64_t ntiles = (W + kTileW - 1) / kTileW;
    const int64_t pmax = static_cast<int64_t>(L) * (N < 256 ? N : 256);
    const size_t plane_bytes = static_cast<size_t>(pmax + 1) * static_cast<size_t>(Wp) * 8;
    if (plane_bytes > (size_t(64) << 30))
        return pc_set_error(ctx, PC_ENOMEM, "pc_eval_selectors: value planes need %zu bytes (L=%d N=%d)", plane_bytes,
                            L, N);
    uint64_t *present, *planes;
    uint32_t *wbase, *prog, *rec, *part;
    int32_t *d_P;
    auto carve = [&](Carver &cv) {
        present = cv.take<uint64_t>(static_cast<size_t>(L) * 4 + 1);
        wbase = cv.take<uint32_t>(static_cast<size_t>(L) * 4 + 1);
        planes = cv.take<uint64_t>(static_cast<size_t>(pmax + 1) * Wp + 2);  // + the all-zero plane pmax
        prog = cv.take<uint32_t>(static_cast<size_t>(n_preds) * 4 + 4);
        rec = cv.take<uint32_t>(static_cast<size_t>(I) * kRecWords + kRecWords);
        part = ntiles > 1 ? cv.take<uint32_t>(static_cast<size_t>(ntiles) * I + 1) : nullptr;
        d_P = cv.take<int32_t>(1);
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    launch_fill_u64(present, static_cast<size_t>(L) * 4, 0, stream);
    if (Wp > 0) launch_fill_u64(planes + static_cast<size_t>(pmax) * Wp, static_cast<size_t>(Wp), 0, stream);
    if (W == 0) launch_fill_u32(popcnt, static_cast<size_t>(I), 0, stream);
    PC_LAUNCH_CHECK(ctx);
    if (N > 0 && L > 0) {
        // about 2048 workgroups: a few hundred nodes each
        const int64_t ltiles = (L + 63) / 64;
        int64_t chunk = (static_cast<int64_t>(N) * ltiles + 2047) / 2048;
        chunk = chunk < 64 ? 64 : (chunk + 3) / 4 * 4;
        while ((N + chunk - 1) / chunk > 65535) chunk *= 2;
        dim3 gp((L + 63) / 64, static_cast<unsigned>((N + chunk - 1) / chunk));
        PC_TIMED(ctx, "k_sel_presence", stream,
                 hipLaunchKernelGGL(k_sel_presence, gp, dim3(256), 0, stream, labels, N, L, chunk,
                                    reinterpret_cast<uint32_t *>(present)));
        PC_LAUNCH_CHECK(ctx);
    }
    if (L > 0) {
        PC_TIMED(ctx, "k_sel_label_scan", stream,
                 hipLaunchKernelGGL(k_sel_label_scan, dim3(1), dim3(1024), 0, stream, present, L, wbase, d_P));
        PC_LAUNCH_CHECK(ctx);
    }
    if (N > 0 && L > 0) {
        dim3 gb(static_cast<unsigned>(W), static_cast<unsigned>((L + 3) / 4));
        PC_TIMED(ctx, "k_sel_planes", stream,
                 hipLaunchKernelGGL(k_sel_planes, gb, dim3(256), 0, stream, labels, N, L, present, wbase, planes, Wp));
        PC_LAUNCH_CHECK(ctx);
    }
    const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>((I + 255) / 256, 8192));
    PC_TIMED(ctx, "k_sel_compile", stream,
             hipLaunchKernelGGL(k_sel_compile, dim3(rgrid), dim3(256), 0, stream, pred_off, preds, n_preds, I, L,
                                present, wbase, static_cast<uint32_t>(pmax), prog, rec, ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    if (W == 0) return PC_OK;

    // about 4096 workgroups; a chunk is a whole number of 256-row passes
    int64_t nchunks = std::max<int64_t>((4096 + ntiles - 1) / ntiles, 1);
    int64_t rpc = (I + nchunks - 1) / nchunks;
    rpc = (rpc + kEvalThreads - 1) / kEvalThreads * kEvalThreads;
    nchunks = (I + rpc - 1) / rpc;
    const int64_t total = ntiles * nchunks;
    const unsigned blocks = static_cast<unsigned>(8 * ((total + 7) / 8));
    uint32_t *cnt_out = ntiles > 1 ? part : popcnt;
    const int64_t pbytes = static_cast<int64_t>(pmax + 1) * Wp * 8;
    auto eval = [&](auto kern) {
        PC_TIMED(ctx, "k_sel_eval", stream,
                 hipLaunchKernelGGL(kern, dim3(blocks), dim3(kEvalThreads), 0, stream, rec, prog, pred_off, preds,
                                    present, wbase, planes, pbytes, Wp, I, static_cast<int32_t>(W), N, feasible,
                                    cnt_out, static_cast<int32_t>(ntiles), static_cast<int32_t>(nchunks),
                                    static_cast<int32_t>(rpc)));
    };
    if (pbytes < (int64_t(1) << 31)) eval(k_sel_eval<true>);  // buffer offsets are 32-bit
    else eval(k_sel_eval<false>);
    PC_LAUNCH_CHECK(ctx);
    if (ntiles > 1) {
        PC_TIMED(ctx, "k_sel_popsum", stream,
                 hipLaunchKernelGGL(k_sel_popsum, dim3(static_cast<unsigned>((I + 255) / 256)), dim3(256), 0, stream,
                                    part, I, static_cast<int32_t>(ntiles), popcnt));
        PC_LAUNCH_CHECK(ctx);
    }
    return PC_OK;
}

// A1 -- placement constraints: node-selector evaluation for every selector
// row x node, emitting a feasible-node bitset and a popcount per row.
//
// The operators are Kubernetes node-affinity's (In / NotIn / Exists over a
// label), which is how the paper compiles a placement constraint such as a
// residency region that the pod's node must carry as a label (Formal Model
// and Satisfaction, example; Service Placement Module).
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
//                  (L2 hits: a tile of every plane is P KiB), exactly as
//                  many as its program has entries, all go out together
//                  with scalar offsets, followed by one output store.  A
//                  row's tiles are shifted so that stores cover whole
//                  128-byte lines.  Per-lane popcounts are collected as
//                  bytes in LDS and summed once per 64 rows; a last pass
//                  sums the tiles.
#include <algorithm>
#include <mutex>
#include <type_traits>

#include "pc_internal.h"

namespace {

constexpr int kEvalThreads = 256;  // 4 wavefronts, one row at a time each
constexpr int kWpl = 2;            // 64-bit words per lane
constexpr int kTileW = 64 * kWpl;  // words per tile
constexpr int kRecWords = 16;      // row record: header + 15 inline entries
constexpr int kInline = kRecWords - 1;
constexpr int kGroup = 8;          // plane loads in flight together
constexpr int kPad = 16;           // plane rows: words before column 0 (a row's shift is at most 15 words)

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
// Word w of plane p lives at planes[p * Wp + kPad + w].
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
    uint64_t *col = planes + kPad + w;
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

// Program entries: plane id, plus flags on the last entry of a clause
// (kLast, kNeg) and, in affinity programs, on the last entry of a term.
constexpr uint32_t kTermEnd = 1u << 29;
constexpr uint32_t kLast = 1u << 30;
constexpr uint32_t kNeg = 1u << 31;
constexpr uint32_t kPidMask = kTermEnd - 1;
// Row record header (word 0); words 1..15 hold an inline program.
constexpr int32_t kRowFalse = -1;     // some clause admits no node (or a malformed predicate)
constexpr int32_t kRowIndirect = -2;  // program of more than 15 entries at prog[4 * word1], word2 entries
constexpr int32_t kRowLong = -3;      // program longer than 4 entries per predicate: decoded on the fly

__device__ __forceinline__ uint32_t plane_id(const uint64_t *pres, const uint32_t *wb, uint32_t v)
{
    const uint32_t k = v >> 6;
    return wb[k] + __popcll(pres[k] & ((1ull << (v & 63)) - 1));
}

// Values lo..hi (clipped to 0..254) as a 256-bit set.
__device__ __forceinline__ void value_range(int64_t lo, int64_t hi, uint64_t s[4])
{
    lo = lo < 0 ? 0 : lo;
    hi = hi > 254 ? 254 : hi;
    for (int k = 0; k < 4; ++k) {
        const int64_t a = lo > 64 * k ? lo : 64 * k;
        const int64_t b = hi < 64 * k + 63 ? hi : 64 * k + 63;
        if (a > b) {
            s[k] = 0;
        } else {
            const int n = static_cast<int>(b - a + 1);
            s[k] = (n == 64 ? ~0ull : ((1ull << n) - 1)) << (a - 64 * k);
        }
    }
}

// The value set a clause ORs over, and whether the OR is negated, for an
// expression with operator op.  Each label value of a node lies in exactly
// one present plane (the absent value 255 included), so In S = OR(S) =
// NOT OR(present \ S) and NotIn S = NOT OR(S) = OR(present \ S): the
// shorter form is taken.  Exists = NOT OR(plane of the absent value), an
// empty OR when every node carries the label; DoesNotExist = that OR.
// Gt t / Lt t are In of the values above / below t.
__device__ __forceinline__ uint32_t expr_clause(uint32_t op, const uint64_t vals[4], const uint64_t *pres,
                                                uint64_t sel[4], bool &neg)
{
    if (op == PC_OP_EXISTS || op == PC_OP_DOESNOTEXIST) {
        sel[0] = sel[1] = sel[2] = 0;
        sel[3] = pres[3] & (1ull << 63);
        neg = op == PC_OP_EXISTS;
        return static_cast<uint32_t>(sel[3] >> 63);
    }
    uint64_t set[4];
    bool is_in = op != PC_OP_NOTIN;
    if (op == PC_OP_GT || op == PC_OP_LT) {
        const int64_t t = static_cast<int64_t>(vals[0]);
        if (op == PC_OP_GT)
            value_range(t >= 254 ? 255 : t + 1, 254, set);
        else
            value_range(0, t <= 0 ? -1 : t - 1, set);
    } else {
        for (int k = 0; k < 4; ++k) set[k] = vals[k];
    }
    uint64_t in[4], out[4];
    uint32_t ms = 0, mc = 0;
    for (int k = 0; k < 4; ++k) {
        in[k] = set[k] & pres[k];
        out[k] = pres[k] & ~set[k];
        ms += __popcll(in[k]);
        mc += __popcll(out[k]);
    }
    const bool use_in = ms <= mc;
    for (int k = 0; k < 4; ++k) sel[k] = use_in ? in[k] : out[k];
    neg = is_in ? !use_in : use_in;
    return use_in ? ms : mc;
}

// The largest present value (0..254, the absent value 255 excluded) at or
// below x, or -1.
__device__ __forceinline__ int32_t pres_max_le(const uint64_t *pres, int64_t x)
{
    if (x < 0) return -1;
    if (x > 254) x = 254;
    const int kx = static_cast<int>(x >> 6);
    for (int k = kx; k >= 0; --k) {
        uint64_t m = pres[k];
        if (k == 3) m &= ~(1ull << 63);
        if (k == kx && (x & 63) != 63) m &= (1ull << ((x & 63) + 1)) - 1;
        if (m) return k * 64 + 63 - __builtin_clzll(m);
    }
    return -1;
}

// Gt / Lt over the label's prefix planes (plane pfx0 + plane_id(v) is the
// OR of the planes of the label's present values <= v, built by
// k_aff_prefix): Lt t is the prefix of the largest present value below t,
// one entry; Gt t is NOT (the prefix of the largest present value <= t OR
// the absent-value plane), at most two entries.  The node sets are those
// expr_clause selects value by value.  Returns the entry count (ids in e)
// with neg as in expr_clause: 0 entries without neg is a clause no node
// satisfies, 0 entries with neg one every node does.
__device__ __forceinline__ uint32_t cmp_clause(uint32_t op, int64_t t, const uint64_t *pres, const uint32_t *wb,
                                               uint32_t pfx0, uint32_t (&e)[2], bool &neg)
{
    uint32_t n = 0;
    neg = false;
    if (op == PC_OP_LT) {
        const int32_t u = t <= 0 ? -1 : pres_max_le(pres, t - 1);
        if (u >= 0) e[n++] = pfx0 + plane_id(pres, wb, static_cast<uint32_t>(u));
        return n;
    }
    const int32_t top = pres_max_le(pres, 254);
    if (top < 0 || t >= top) return 0;  // no present value above t
    neg = true;
    const int32_t u = pres_max_le(pres, t);
    if (u >= 0) e[n++] = pfx0 + plane_id(pres, wb, static_cast<uint32_t>(u));
    if (pres[3] >> 63) e[n++] = plane_id(pres, wb, 255);
    return n;
}

// cmp_clause's entry count and neg, without the plane ids.
__device__ __forceinline__ uint32_t cmp_count(uint32_t op, int64_t t, const uint64_t *pres, bool &neg)
{
    neg = false;
    if (op == PC_OP_LT) return (t > 0 && pres_max_le(pres, t - 1) >= 0) ? 1u : 0u;
    const int32_t top = pres_max_le(pres, 254);
    if (top < 0 || t >= top) return 0;
    neg = true;
    return (pres_max_le(pres, t) >= 0 ? 1u : 0u) + static_cast<uint32_t>(pres[3] >> 63);
}

// The program entries of one affinity expression (label present table
// pres / plane bases wb): Gt / Lt through the prefix planes, the rest value
// by value.  emit(entry) receives each entry, the clause's last with kLast
// and, when the clause is negated, kNeg.  Returns the count and the
// clause's emptiness as expr_clause does (count 0 without neg: no node).
template <class Emit>
__device__ __forceinline__ uint32_t aff_entries(const pc_pred &q, const uint64_t *pres, const uint32_t *wb,
                                                uint32_t pfx0, bool &neg, const Emit &emit)
{
    if (q.op == PC_OP_GT || q.op == PC_OP_LT) {
        uint32_t e[2];
        const uint32_t n = cmp_clause(q.op, static_cast<int64_t>(q.vals[0]), pres, wb, pfx0, e, neg);
        for (uint32_t i = 0; i < n; ++i) emit(e[i] | (i + 1 == n ? kLast | (neg ? kNeg : 0u) : 0u));
        return n;
    }
    uint64_t sel[4];
    uint32_t cnt = expr_clause(q.op, q.vals, pres, sel, neg);
    const uint32_t n = cnt;
    for (int k = 0; k < 4; ++k) {
        uint64_t m = sel[k];
        while (m) {
            const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
            m &= m - 1;
            uint32_t ent = plane_id(pres, wb, v);
            if (--cnt == 0) ent |= kLast | (neg ? kNeg : 0u);
            emit(ent);
        }
    }
    return n;
}

__device__ __forceinline__ uint32_t pred_clause(const pc_pred &q, const uint64_t *pres, uint64_t sel[4], bool &neg)
{
    return expr_clause(q.op, q.vals, pres, sel, neg);
}

// Well-formed affinity expression: label < L, op <= 5, reserved fields 0,
// no value 255 in an In / NotIn set, vals[1..3] = 0 for Gt / Lt.
__device__ __forceinline__ bool aff_valid(const pc_pred &q, int32_t L)
{
    if (static_cast<int32_t>(q.label) >= L || q.op > PC_OP_LT || q.rsv0 != 0 || q.rsv1 != 0) return false;
    if (q.op <= PC_OP_NOTIN && (q.vals[3] >> 63)) return false;
    if ((q.op == PC_OP_GT || q.op == PC_OP_LT) && (q.vals[1] | q.vals[2] | q.vals[3])) return false;
    return true;
}

// One thread per row, two passes over its predicates: validate and size
// the program, then emit it -- inline in the row record when it has at most
// 15 entries, else at prog[4 * pred_off[i] ...] (at most 4 entries per
// predicate; longer programs are decoded at evaluation time).
// One thread per row.  Each row's record is built in LDS and written as
// four 16-byte stores instead of a store per entry.  (Staging a pass's
// predicates in LDS as well measured slower: the 50 KB it takes leaves two
// workgroups per CU.)
constexpr int kCompThreads = 256;
__global__ __launch_bounds__(kCompThreads) void k_sel_compile(const int32_t *__restrict__ pred_off,
                                                              const pc_pred *__restrict__ preds, int64_t n_preds,
                                                              int32_t I, int32_t L,
                                                              const uint64_t *__restrict__ present,
                                                              const uint32_t *__restrict__ wbase,
                                                              uint32_t *__restrict__ prog, uint32_t *__restrict__ rec,
                                                              uint32_t *__restrict__ d_err)
{
    __shared__ uint32_t srec[kCompThreads][kRecWords + 1];  // each thread's row record (padded row)
    uint32_t *R = srec[threadIdx.x];
    uint32_t errs = 0;
    for (int64_t i0 = static_cast<int64_t>(blockIdx.x) * kCompThreads; i0 < I;
         i0 += static_cast<int64_t>(gridDim.x) * kCompThreads) {
        const int64_t i = i0 + threadIdx.x;
        if (i >= I) continue;
        const int64_t b = pred_off[i], e = pred_off[i + 1];
        // the row's record, in LDS until it is complete
        [&] {
            if (!pc_range_ok(b, e, n_preds)) {
                errs |= PC_DERR_OFFSETS;
                R[0] = static_cast<uint32_t>(kRowFalse);
                return;
            }
            // one pass: validity, sizes and the inline entries together
            // (counted past the inline area; a longer program is written
            // again into prog below)
            bool empty = false;
            int64_t n = 0;
            auto emit = [&](const pc_pred &q, uint32_t *out, int64_t &k_out, bool bounded) {
                const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
                const uint32_t *wb = wbase + static_cast<int64_t>(q.label) * 4;
                uint64_t sel[4];
                bool neg;
                const uint32_t cnt0 = pred_clause(q, pres, sel, neg);
                uint32_t cnt = cnt0;
                for (int k = 0; k < 4; ++k) {
                    uint64_t m = sel[k];
                    while (m) {
                        const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                        m &= m - 1;
                        uint32_t ent = plane_id(pres, wb, v);
                        if (--cnt == 0) ent |= kLast | (neg ? kNeg : 0u);
                        if (!bounded || k_out < kInline) out[k_out] = ent;
                        ++k_out;
                    }
                }
                return cnt0 == 0 && !neg;  // an empty OR: no node (a negated empty OR is every node)
            };
            int64_t k_in = 0;
            for (int64_t p = b; p < e; ++p) {
                const pc_pred q = preds[p];
                if (!pred_valid(q.label, q.op, q.rsv0, q.rsv1, q.vals[3], L)) {
                    errs |= PC_DERR_PRED;
                    empty = true;
                    continue;
                }
                if (empty) continue;
                if (emit(q, R + 1, k_in, true)) empty = true;
            }
            n = k_in;
            if (empty) {
                R[0] = static_cast<uint32_t>(kRowFalse);
                return;
            }
            if (n <= kInline) {
                R[0] = static_cast<uint32_t>(n);  // the evaluator reads entries 1..n only
                return;
            }
            if (n > 4 * (e - b)) {
                R[0] = static_cast<uint32_t>(kRowLong);
                return;
            }
            int64_t k_out = 0;
            for (int64_t p = b; p < e; ++p) emit(preds[p], prog + 4 * b, k_out, false);
            R[0] = static_cast<uint32_t>(kRowIndirect);
            R[1] = static_cast<uint32_t>(b);
            R[2] = static_cast<uint32_t>(n);
        }();
        uint4 *dst = reinterpret_cast<uint4 *>(rec + i * kRecWords);
#pragma unroll
        for (int k = 0; k < kRecWords / 4; ++k) dst[k] = make_uint4(R[4 * k], R[4 * k + 1], R[4 * k + 2], R[4 * k + 3]);
    }
    if (errs) atomicOr(d_err, errs);
}

// Affinity input sweep: the data-error flags are properties of the whole
// input.  OFFSETS for any bad term or row offset pair, PRED for any
// malformed expression inside a term with a valid offset pair.
__global__ __launch_bounds__(256) void k_aff_validate(const int32_t *__restrict__ row_off, int32_t I,
                                                      const int32_t *__restrict__ term_off, int32_t n_terms,
                                                      const pc_pred *__restrict__ preds, int64_t n_preds, int32_t L,
                                                      uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    const int64_t tot = I > n_terms ? I : n_terms;
    for (int64_t x = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; x < tot;
         x += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (x < n_terms) {
            const int64_t b = term_off[x], e = term_off[x + 1];
            if (!pc_range_ok(b, e, n_preds)) {
                errs |= PC_DERR_OFFSETS;
            } else {
                for (int64_t p = b; p < e; ++p)
                    if (!aff_valid(preds[p], L)) {
                        errs |= PC_DERR_PRED;
                        break;
                    }
            }
        }
        if (x < I && !pc_range_ok(row_off[x], row_off[x + 1], n_terms)) errs |= PC_DERR_OFFSETS;
    }
    if (errs) atomicOr(d_err, errs);
}

// Inventory flags of one well-formed expression: its label carries no
// value on any node, or an In / NotIn value no node carries.
__device__ __forceinline__ uint32_t aff_unknown(const pc_pred &q, const uint64_t *pres)
{
    uint32_t u = 0;
    if ((pres[0] | pres[1] | pres[2] | (pres[3] & ~(1ull << 63))) == 0) u |= PC_UNKNOWN_KEY;
    if (q.op <= PC_OP_NOTIN &&
        ((q.vals[0] & ~pres[0]) | (q.vals[1] & ~pres[1]) | (q.vals[2] & ~pres[2]) | (q.vals[3] & ~pres[3])))
        u |= PC_UNKNOWN_VALUE;
    return u;
}

// Whether term [b, e) can hold for some node at all (valid offsets, at
// least one expression, every expression well-formed, no clause that is an
// empty OR), and its program length (Gt / Lt in the prefix form).
__device__ __forceinline__ bool aff_term(const pc_pred *__restrict__ preds, int64_t b, int64_t e, int64_t n_preds,
                                         int32_t L, const uint64_t *__restrict__ present, int64_t &len)
{
    len = 0;
    if (!pc_range_ok(b, e, n_preds) || b == e) return false;
    bool ok = true;
    for (int64_t p = b; p < e; ++p) {
        const pc_pred q = preds[p];
        if (!aff_valid(q, L)) return false;
        const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
        bool neg;
        uint32_t cnt;
        if (q.op == PC_OP_GT || q.op == PC_OP_LT) {
            cnt = cmp_count(q.op, static_cast<int64_t>(q.vals[0]), pres, neg);
        } else {
            uint64_t sel[4];
            cnt = expr_clause(q.op, q.vals, pres, sel, neg);
        }
        if (cnt == 0 && !neg) ok = false;
        len += cnt;
    }
    return ok;
}

// One thread per affinity row: inventory flags, then the program.  Terms
// that hold nowhere are dropped; a term with an empty program holds
// everywhere, and so does a row without terms (header 0); a row with no
// term left admits no node.  The last entry of each term carries
// kTermEnd.  Programs of at most 15 entries sit inline in the row record;
// longer ones take a slice of prog through a bump counter and, when it is
// exhausted, are decoded at evaluation time (kRowLong).
__global__ __launch_bounds__(256) void k_aff_compile(const int32_t *__restrict__ row_off, int32_t I,
                                                     const int32_t *__restrict__ term_off, int32_t n_terms,
                                                     const pc_pred *__restrict__ preds, int64_t n_preds, int32_t L,
                                                     const uint64_t *__restrict__ present,
                                                     const uint32_t *__restrict__ wbase,
                                                     uint32_t *__restrict__ prog, int64_t prog_cap,
                                                     unsigned long long *__restrict__ prog_used,
                                                     uint32_t *__restrict__ rec, uint8_t *__restrict__ unknown,
                                                     uint32_t pfx0)
{
    // each row's record is built in LDS and written as 16-byte stores
    __shared__ uint32_t srec[256][kRecWords + 1];
    uint32_t *rr = srec[threadIdx.x];
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < I; i += gridDim.x * blockDim.x) {
        [&] {  // the row's record, in LDS until it is complete
            const int64_t tb = row_off[i], te = row_off[i + 1];
            if (!pc_range_ok(tb, te, n_terms)) {
                rr[0] = static_cast<uint32_t>(kRowFalse);
                unknown[i] = 0;
                return;
            }
            // One pass over the row's expressions: the inventory flags (every
            // well-formed expression of every term with valid offsets), and
            // each term's entries emitted into the record's inline area as
            // they come (counted past its end) and taken back when the term
            // turns out to hold nowhere (a malformed expression, an empty
            // clause).  A live term with no entries holds everywhere, and so
            // does the row.
            uint32_t unk = 0;
            bool all = tb == te;
            int64_t n = 0, live = 0, k_out = 0;
            uint32_t *in_out = rr + 1;
            for (int64_t t = tb; t < te; ++t) {
                const int64_t b = term_off[t], e = term_off[t + 1];
                if (!pc_range_ok(b, e, n_preds)) continue;
                bool ok = b != e;
                const int64_t start = k_out;
                int64_t len = 0;
                for (int64_t p = b; p < e; ++p) {
                    const pc_pred q = preds[p];
                    if (!aff_valid(q, L)) {
                        ok = false;
                        continue;
                    }
                    const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
                    unk |= aff_unknown(q, pres);
                    if (!ok || all) continue;
                    bool neg;
                    const uint32_t cnt = aff_entries(q, pres, wbase + static_cast<int64_t>(q.label) * 4, pfx0, neg,
                                                     [&](uint32_t ent) {
                                                         if (k_out < kInline) in_out[k_out] = ent;
                                                         ++k_out;
                                                     });
                    if (cnt == 0 && !neg) ok = false;
                    len += cnt;
                }
                if (all) continue;
                if (!ok) {
                    k_out = start;
                    continue;
                }
                if (len == 0) {
                    all = true;
                    continue;
                }
                if (k_out <= kInline) in_out[k_out - 1] |= kTermEnd;
                n += len;
                ++live;
            }
            unknown[i] = static_cast<uint8_t>(unk);
            if (all) {
                rr[0] = 0;
                return;
            }
            if (live == 0) {
                rr[0] = static_cast<uint32_t>(kRowFalse);
                return;
            }
            if (n <= kInline) {
                rr[0] = static_cast<uint32_t>(n);
                return;
            }
            // longer than the inline area: a slice of prog, written by a
            // second pass (slices are whole multiples of 4 entries: the
            // record stores off / 4)
            const unsigned long long off = atomicAdd(prog_used, static_cast<unsigned long long>((n + 3) & ~int64_t(3)));
            if (static_cast<int64_t>(off) + n > prog_cap) {
                rr[0] = static_cast<uint32_t>(kRowLong);
                return;
            }
            uint32_t *out = prog + off;
            rr[0] = static_cast<uint32_t>(kRowIndirect);
            rr[1] = static_cast<uint32_t>(off / 4);
            rr[2] = static_cast<uint32_t>(n);
            int64_t k2 = 0;
            for (int64_t t = tb; t < te; ++t) {
                const int64_t b = term_off[t], e = term_off[t + 1];
                int64_t len;
                if (!aff_term(preds, b, e, n_preds, L, present, len)) continue;
                for (int64_t p = b; p < e; ++p) {
                    const pc_pred q = preds[p];
                    bool neg;
                    aff_entries(q, present + static_cast<int64_t>(q.label) * 4, wbase + static_cast<int64_t>(q.label) * 4,
                                pfx0, neg, [&](uint32_t ent) { out[k2++] = ent; });
                }
                out[k2 - 1] |= kTermEnd;
            }
        }();
        uint4 *dst = reinterpret_cast<uint4 *>(rec + static_cast<int64_t>(i) * kRecWords);
#pragma unroll
        for (int k = 0; k < kRecWords / 4; ++k)
            dst[k] = make_uint4(rr[4 * k], rr[4 * k + 1], rr[4 * k + 2], rr[4 * k + 3]);
    }
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
// In affinity programs (kTerms) the end of a term ORs the term's
// conjunction into the row (r) and starts the next term.
template <bool kTerms>
__device__ __forceinline__ void fold(uint32_t ent, const Words &v, Words &c, Words &a, Words &r)
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
    if constexpr (kTerms) {
        if (ent & kTermEnd) {
            r.a |= a.a;
            r.b |= a.b;
            a.a = a.b = ~0ull;
        }
    }
}

// This lane's two words of plane `pid`.  The buffer form (planes within
// 4 GiB) takes the plane offset as a scalar operand: one scalar multiply
// per load and no vector address arithmetic.
template <bool kBuf>
struct Planes {
    __amdgpu_buffer_rsrc_t rsrc;
    uint32_t lane_off;  // bytes: this lane's first word within a plane row (set per row)
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

// Affinity rows whose program found no slice: the terms decoded on the
// scalar unit (the same term rules as k_aff_compile).
template <bool kBuf>
__device__ Words eval_row_decoded_aff(const pc_pred *__restrict__ preds, int64_t n_preds,
                                      const int32_t *__restrict__ term_off, int64_t tb, int64_t te, int32_t L,
                                      const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
                                      const Planes<kBuf> &pl)
{
    Words r{0, 0};
    for (int64_t t = tb; t < te; ++t) {
        int64_t len;
        const int64_t b = term_off[t], e = term_off[t + 1];
        if (!aff_term(preds, b, e, n_preds, L, present, len)) continue;
        Words a{~0ull, ~0ull};
        for (int64_t p = b; p < e; ++p) {
            const pc_pred q = preds[p];
            const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
            const uint32_t *wb = wbase + static_cast<int64_t>(q.label) * 4;
            uint64_t sel[4];
            bool neg;
            expr_clause(q.op, q.vals, pres, sel, neg);
            Words c{0, 0};
            for (int k = 0; k < 4; ++k) {
                uint64_t m = sel[k];
                while (m) {
                    const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                    m &= m - 1;
                    const Words x = pl(plane_id(pres, wb, v));
                    c.a |= x.a;
                    c.b |= x.b;
                }
            }
            a.a &= neg ? ~c.a : c.a;
            a.b &= neg ? ~c.b : c.b;
        }
        r.a |= a.a;
        r.b |= a.b;
    }
    return r;
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
// kTerms: affinity rows (pred_off holds the row -> term offsets, term_off
// the term -> expression offsets) whose programs OR their terms.  kStore
// false: popcounts only, no bitset written (verdict-only runs).
template <bool kBuf, bool kTerms, bool kStore = true>
__global__ __launch_bounds__(kEvalThreads) void k_sel_eval(
    const uint32_t *__restrict__ rec, const uint32_t *__restrict__ prog, const int32_t *__restrict__ pred_off,
    const pc_pred *__restrict__ preds, const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
    const uint64_t *__restrict__ planes, int64_t plane_bytes, int64_t Wp, int32_t I, int32_t W, int32_t N,
    uint64_t *__restrict__ feasible, uint32_t *__restrict__ part, int32_t ntiles, int32_t nchunks, int32_t rpc,
    const int32_t *__restrict__ term_off, int64_t n_preds, int32_t L, int32_t shift)
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
    const int32_t wt = tile * kTileW + lane * kWpl;  // this lane's first word of an unshifted row
    const uint64_t last = (N & 63) ? (1ull << (N & 63)) - 1 : ~0ull;
    // word index of the bitset's start within its 128-byte line
    const uint32_t base16 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(feasible) >> 3) & 15u;
    Planes<kBuf> pl;
    if constexpr (kBuf)
        pl.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(planes), static_cast<short>(0),
                                                    static_cast<int>(plane_bytes), 0x00020000);
    pl.rowbytes = static_cast<uint32_t>(Wp * 8);
    pl.Wp = Wp;
    // Per-row geometry.  With shift on, the tiles of row r start s(r) words
    // early, where s(r) is the row start's word offset within its 128-byte
    // line: every store then covers whole lines except at the row's two
    // ends, instead of splitting a line between two tiles at every tile
    // edge.  Lanes outside [0, W) load pad words of the plane rows and are
    // masked.
    int32_t w0 = 0;
    bool ok0 = false, ok1 = false, pair = false;
    uint64_t m0 = 0, m1 = 0;
    auto geom = [&](int32_t r) {
        const uint32_t rw = (static_cast<uint32_t>(r) & 15u) * (static_cast<uint32_t>(W) & 15u);  // r * W mod 16
        const int32_t sh = shift ? static_cast<int32_t>((base16 + rw) & 15u) : 0;
        w0 = wt - sh;
        ok0 = w0 >= 0 && w0 < W;
        ok1 = w0 + 1 >= 0 && w0 + 1 < W;
        m0 = ok0 ? (w0 == W - 1 ? last : ~0ull) : 0ull;
        m1 = ok1 ? (w0 + 1 == W - 1 ? last : ~0ull) : 0ull;
        pair = ok0 && ok1 && ((base16 + rw + static_cast<uint32_t>(w0)) & 1u) == 0;  // 16-byte aligned pair
        pl.lane_off = static_cast<uint32_t>(kPad + w0) * 8u;
        pl.pcol = planes + kPad + w0;
    };
    uint8_t *cb = reinterpret_cast<uint8_t *>(cnt_lds[wave]);
    uint32_t *prt = part + static_cast<int64_t>(tile) * I;
    const int32_t r0 = chunk * rpc;
    const int32_t r1 = min(I, r0 + rpc);
    // One row: its record R (uniform, in SGPRs) -> bitset store and count
    // byte.  kIn: an interior tile of a line-shifted row (every lane's two
    // words lie in [0, W - 1), so no masks, and every pair is 16-byte
    // aligned); its geometry is one subtraction per lane.
    const uint32_t lane_base = static_cast<uint32_t>(kPad + wt) * 8u;
    auto row_shift = [&](int32_t r) {
        const uint32_t rw = (static_cast<uint32_t>(r) & 15u) * (static_cast<uint32_t>(W) & 15u);  // r * W mod 16
        return shift ? static_cast<int32_t>((base16 + rw) & 15u) : 0;
    };
    auto row = [&](auto in_tag, int32_t r, int32_t i, const uint32_t (&R)[kRecWords]) {
        constexpr bool kIn = decltype(in_tag)::value;
        const int32_t hdr = static_cast<int32_t>(R[0]);
        if constexpr (kIn) {
            const int32_t sh = row_shift(r);
            w0 = wt - sh;
            pl.lane_off = lane_base - static_cast<uint32_t>(sh) * 8u;
            if constexpr (!kBuf) pl.pcol = planes + kPad + w0;
        } else {
            geom(r);
        }
        Words a{~0ull, ~0ull};
        Words rt{0, 0};  // affinity: OR of the finished terms
        if (hdr == kRowFalse) {
            a = Words{0, 0};
        } else if (hdr > 0) {
            // inline program of hdr entries: the length is uniform, so the
            // guards are scalar branches and only real entries are loaded
            Words c{0, 0};
            {
                Words V[kGroup];
#pragma unroll
                for (int k = 0; k < kGroup; ++k)
                    if (k < hdr) V[k] = pl(R[1 + k] & kPidMask);
#pragma unroll
                for (int k = 0; k < kGroup; ++k)
                    if (k < hdr) fold<kTerms>(R[1 + k], V[k], c, a, rt);
            }
            if (hdr > kGroup) {
                Words V[kInline - kGroup];
#pragma unroll
                for (int k = 0; k < kInline - kGroup; ++k)
                    if (kGroup + k < hdr) V[k] = pl(R[1 + kGroup + k] & kPidMask);
#pragma unroll
                for (int k = 0; k < kInline - kGroup; ++k)
                    if (kGroup + k < hdr) fold<kTerms>(R[1 + kGroup + k], V[k], c, a, rt);
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
                    if (e0 + k < len) fold<kTerms>(E[k], V[k], c, a, rt);
            }
        } else if (hdr == kRowLong) {
            if constexpr (kTerms)
                rt = eval_row_decoded_aff<kBuf>(preds, n_preds, term_off, pred_off[r], pred_off[r + 1], L, present,
                                                wbase, pl);
            else
                a = eval_row_decoded<kBuf>(preds, pred_off[r], pred_off[r + 1], present, wbase, pl);
        }
        if constexpr (kTerms) {
            if (hdr > 0 || hdr == kRowIndirect || hdr == kRowLong) a = rt;
        }
        if constexpr (!kIn) {
            a.a &= m0;
            a.b &= m1;
        }
        if constexpr (kStore) {
            const int64_t at = static_cast<int64_t>(r) * W + w0;
            if (kIn || pair) {
                __builtin_nontemporal_store(u64x2{a.a, a.b}, reinterpret_cast<u64x2 *>(feasible + at));
            } else {
                if (ok0) __builtin_nontemporal_store(a.a, feasible + at);
                if (ok1) __builtin_nontemporal_store(a.b, feasible + at + 1);
            }
        }
        cb[i * kCntStride + lane] = static_cast<uint8_t>(__popcll(a.a) + __popcll(a.b));
    };
    // (affinity programs measured slower with the interior path: it is
    // taken for selector rows only)
    auto row_any = [&](int32_t r, int32_t i, const uint32_t (&R)[kRecWords]) {
        const int32_t lo = tile * kTileW - row_shift(r);
        if (!kTerms && shift && lo >= 0 && lo + kTileW <= W - 1) row(std::true_type{}, r, i, R);
        else row(std::false_type{}, r, i, R);
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
            row_any(bat + i, i, RA);
            if (i + 1 < nb) {
                load_rec(bat + min(i + 2, nb - 1), RA);
                row_any(bat + i + 1, i + 1, RB);
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

// ---------------------------------------------------------------- preferred
// Preferred node affinity: per row, weighted terms (weight 1..100, terms as
// in required affinity); a node's score is the sum of the weights of the
// terms that hold for it; the best feasible node has the largest score, the
// lowest index among equal scores.  Scores are kept bit-sliced: bit b of
// every node's score of a 64-node word is one 64-bit word, so adding a
// term's weight to the nodes where it holds is a ripple add over the score
// bits, and the maximum over a word's nodes is found from the top bit down.
constexpr int kScoreBits = 16;         // 655 terms of weight <= 100 stay below 2^16
constexpr int32_t kPrefMaxTerms = 655;
constexpr uint32_t kPrefLenBits = 24;  // term header: weight << 24 | program entries
// row record, 16 words (one 64-byte line): word 0 = kind << 24 | score bits
// << 16 | live terms; word 1 = program offset in prog (kPrefIndirect);
// words 2..15 = the program itself when it has at most 14 words
enum : uint32_t { kPrefInline = 0, kPrefIndirect = 1, kPrefDecode = 2, kPrefNone = 3 };
constexpr int kPrefRec = 16;
constexpr int kPrefInlineWords = kPrefRec - 2;
constexpr uint32_t kPrefClasses = 4;  // row lists: scores within 8 bits, within 16 bits, decoded, <= 3 terms
constexpr uint32_t kPrefFewTerms = 3;  // rows with at most this many live terms: scores from term patterns

__device__ __forceinline__ bool pref_weight_ok(uint32_t w) { return w >= 1 && w <= 100; }

__device__ __forceinline__ bool pref_row_ok(const int32_t *__restrict__ row_off, int64_t i, int32_t n_terms)
{
    const int64_t b = row_off[i], e = row_off[i + 1];
    return pc_range_ok(b, e, n_terms) && e - b <= kPrefMaxTerms;
}

__device__ __forceinline__ uint32_t bit_length(uint32_t x) { return x ? 32u - __builtin_clz(x) : 0u; }

// Input sweep: the data-error flags are properties of the whole input.
// PRED for a weight outside 1..100 or a malformed expression inside a term
// with a valid offset pair; OFFSETS for a bad term or row offset pair or a
// row of more than kPrefMaxTerms terms.
__global__ __launch_bounds__(256) void k_pref_validate(const int32_t *__restrict__ row_off, int32_t I,
                                                       const int32_t *__restrict__ term_off, int32_t n_terms,
                                                       const uint32_t *__restrict__ weight,
                                                       const pc_pred *__restrict__ preds, int64_t n_preds, int32_t L,
                                                       uint32_t *__restrict__ d_err)
{
    uint32_t errs = 0;
    const int64_t tot = I > n_terms ? I : n_terms;
    for (int64_t x = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; x < tot;
         x += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        if (x < n_terms) {
            if (!pref_weight_ok(weight[x])) errs |= PC_DERR_PRED;
            const int64_t b = term_off[x], e = term_off[x + 1];
            if (!pc_range_ok(b, e, n_preds)) {
                errs |= PC_DERR_OFFSETS;
            } else {
                for (int64_t p = b; p < e; ++p)
                    if (!aff_valid(preds[p], L)) {
                        errs |= PC_DERR_PRED;
                        break;
                    }
            }
        }
        if (x < I && !pref_row_ok(row_off, x, n_terms)) errs |= PC_DERR_OFFSETS;
    }
    if (errs) atomicOr(d_err, errs);
}

// One row of k_pref_compile: its record, and its class (3: at most three
// live terms, including none; 0: scores fit 8 bits, 1: 16 bits; 2: decoded
// on the fly).
__device__ uint32_t pref_compile_row(const int32_t *__restrict__ row_off, int32_t i,
                                     const int32_t *__restrict__ term_off, int32_t n_terms,
                                     const uint32_t *__restrict__ weight, const pc_pred *__restrict__ preds,
                                     int64_t n_preds, int32_t L, const uint64_t *__restrict__ present,
                                     const uint32_t *__restrict__ wbase, uint32_t *__restrict__ prog, int64_t prog_cap,
                                     unsigned long long *__restrict__ prog_used, uint32_t *rr, uint32_t pfx0)
{
    rr[0] = kPrefNone << 24;
    if (!pref_row_ok(row_off, i, n_terms)) return 3;
    const int64_t tb = row_off[i], te = row_off[i + 1];
    // One pass: each live term's header and entries go into the record's
    // inline words as they come (counted past their end); a term that turns
    // out dead (weight out of range, a malformed expression, an empty
    // clause) is taken back.  Programs past the inline words are written
    // again, into a slice of prog.
    int64_t n = 0, k_out = 0;
    uint32_t live = 0, sum = 0;
    bool decode = false;
    uint32_t *in_out = rr + 2;
    auto put = [&](uint32_t word) {
        if (k_out < kPrefInlineWords) in_out[k_out] = word;
        ++k_out;
    };
    for (int64_t t = tb; t < te; ++t) {
        const uint32_t w = weight[t];
        const int64_t b = term_off[t], e = term_off[t + 1];
        if (!pref_weight_ok(w) || !pc_range_ok(b, e, n_preds) || b == e) continue;
        const int64_t start = k_out;
        put(0u);  // the header, set below
        bool ok = true;
        int64_t len = 0;
        for (int64_t p = b; p < e && ok; ++p) {
            const pc_pred q = preds[p];
            if (!aff_valid(q, L)) {
                ok = false;
                break;
            }
            bool neg;
            const uint32_t cnt = aff_entries(q, present + static_cast<int64_t>(q.label) * 4,
                                             wbase + static_cast<int64_t>(q.label) * 4, pfx0, neg, put);
            if (cnt == 0 && !neg) ok = false;
            len += cnt;
        }
        if (!ok) {
            k_out = start;
            continue;
        }
        if (len >= (int64_t(1) << kPrefLenBits)) decode = true;
        if (start < kPrefInlineWords) in_out[start] = w << kPrefLenBits | static_cast<uint32_t>(len);
        n += 1 + len;
        sum += w;
        ++live;
    }
    if (live == 0) return 3;
    const uint32_t head = live | bit_length(sum) << 16;
    uint32_t kind = kPrefInline;
    if (!decode && n > kPrefInlineWords) {
        const unsigned long long off = atomicAdd(prog_used, static_cast<unsigned long long>(n));
        decode = static_cast<int64_t>(off) + n > prog_cap;
        if (!decode) {
            uint32_t *out = prog + off;
            rr[1] = static_cast<uint32_t>(off);
            kind = kPrefIndirect;
            int64_t k2 = 0;
            for (int64_t t = tb; t < te; ++t) {
                const int64_t b = term_off[t], e = term_off[t + 1];
                int64_t len;
                if (!pref_weight_ok(weight[t]) || !aff_term(preds, b, e, n_preds, L, present, len)) continue;
                out[k2++] = weight[t] << kPrefLenBits | static_cast<uint32_t>(len);
                for (int64_t p = b; p < e; ++p) {
                    const pc_pred q = preds[p];
                    bool neg;
                    aff_entries(q, present + static_cast<int64_t>(q.label) * 4,
                                wbase + static_cast<int64_t>(q.label) * 4, pfx0, neg,
                                [&](uint32_t ent) { out[k2++] = ent; });
                }
            }
        }
    }
    if (decode) {
        rr[0] = head | kPrefDecode << 24;
        return 2;
    }
    rr[0] = head | kind << 24;
    if (live <= kPrefFewTerms) return 3;
    return bit_length(sum) <= 8 ? 0u : 1u;
}

// One thread per row: the row's live terms (weight in range, and able to
// hold somewhere) as a program of term headers, each followed by its clause
// entries (kLast / kNeg as in selector programs), inline in the row record
// when it has at most 14 words, else in a slice of prog taken through a
// bump counter.  When the slice does not fit, or a term has more than 2^24
// entries, the row is decoded at evaluation time.
// Each row is appended to the list of its class.
__global__ __launch_bounds__(256) void k_pref_compile(const int32_t *__restrict__ row_off, int32_t I,
                                                      const int32_t *__restrict__ term_off, int32_t n_terms,
                                                      const uint32_t *__restrict__ weight,
                                                      const pc_pred *__restrict__ preds, int64_t n_preds, int32_t L,
                                                      const uint64_t *__restrict__ present,
                                                      const uint32_t *__restrict__ wbase, uint32_t *__restrict__ prog,
                                                      int64_t prog_cap, unsigned long long *__restrict__ prog_used,
                                                      uint32_t *__restrict__ rec, int32_t *__restrict__ list,
                                                      uint32_t *__restrict__ list_len, uint32_t pfx0)
{
    // each row's record is built in LDS and written as 16-byte stores
    __shared__ uint32_t srec[256][kPrefRec + 1];
    uint32_t *R = srec[threadIdx.x];
    const int lane = threadIdx.x & 63;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * blockDim.x; base < I;
         base += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int32_t i = static_cast<int32_t>(base + threadIdx.x);
        uint32_t cls = kPrefClasses;
        if (i < I) {
            cls = pref_compile_row(row_off, i, term_off, n_terms, weight, preds, n_preds, L, present, wbase, prog,
                                   prog_cap, prog_used, R, pfx0);
            uint4 *dst = reinterpret_cast<uint4 *>(rec + static_cast<int64_t>(i) * kPrefRec);
#pragma unroll
            for (int k = 0; k < kPrefRec / 4; ++k)
                dst[k] = make_uint4(R[4 * k], R[4 * k + 1], R[4 * k + 2], R[4 * k + 3]);
        }
        // append i to its class list: one counter update per class and wavefront
        for (uint32_t c = 0; c < kPrefClasses; ++c) {
            const uint64_t mask = __ballot(cls == c);
            if (mask == 0) continue;
            const int leader = __builtin_ctzll(mask);
            uint32_t off = 0;
            if (lane == leader) off = atomicAdd(list_len + c, static_cast<uint32_t>(__popcll(mask)));
            off = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(off), leader));
            const uint32_t below = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                                             __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
            if (cls == c) list[static_cast<int64_t>(c) * I + off + below] = i;
        }
    }
}


// Wavefront reductions of a 32-bit value with DPP: quad exchanges, then
// row rotations by 4 and 8 leave every lane with its 16-lane row's result;
// the four rows' results are combined on the scalar unit.
template <int kOp>
__device__ __forceinline__ uint32_t red_op(uint32_t a, uint32_t b)
{
    if constexpr (kOp == 0) return a > b ? a : b;
    else if constexpr (kOp == 1) return a < b ? a : b;
    else return a + b;
}

template <int kOp>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t x)
{
    int v = static_cast<int>(x);
    v = static_cast<int>(red_op<kOp>(static_cast<uint32_t>(v), static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false))));
    v = static_cast<int>(red_op<kOp>(static_cast<uint32_t>(v), static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false))));
    v = static_cast<int>(red_op<kOp>(static_cast<uint32_t>(v), static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0x124, 0xF, 0xF, false))));
    v = static_cast<int>(red_op<kOp>(static_cast<uint32_t>(v), static_cast<uint32_t>(__builtin_amdgcn_update_dpp(v, v, 0x128, 0xF, 0xF, false))));
    const uint32_t r0 = static_cast<uint32_t>(__builtin_amdgcn_readlane(v, 0));
    const uint32_t r1 = static_cast<uint32_t>(__builtin_amdgcn_readlane(v, 16));
    const uint32_t r2 = static_cast<uint32_t>(__builtin_amdgcn_readlane(v, 32));
    const uint32_t r3 = static_cast<uint32_t>(__builtin_amdgcn_readlane(v, 48));
    return red_op<kOp>(red_op<kOp>(r0, r1), red_op<kOp>(r2, r3));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) { return wave_reduce_u32<0>(x); }
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) { return wave_reduce_u32<1>(x); }
__device__ __forceinline__ uint32_t wave_add_u32(uint32_t x) { return wave_reduce_u32<2>(x); }

// acc += w * a, bit-sliced over kBits score bits (w <= 100 < 2^7): bits
// 0..6 are full adds of the weight's bit (masked by a) and the carry, above
// them only the carry moves.  The row's class guarantees that its weight
// sum fits kBits, so no carry leaves the top bit.  Branch-free, so the
// score words stay in place.
template <int kBits>
__device__ __forceinline__ void score_add(Words (&acc)[kBits], uint32_t w, const Words &a)
{
    Words carry{0, 0};
#pragma unroll
    for (int b = 0; b < 7; ++b) {
        const uint64_t wm = ((w >> b) & 1u) ? ~0ull : 0ull;
        const uint64_t xa = acc[b].a, xb = acc[b].b, ya = a.a & wm, yb = a.b & wm;
        acc[b].a = xa ^ ya ^ carry.a;
        acc[b].b = xb ^ yb ^ carry.b;
        carry.a = (xa & ya) | (carry.a & (xa ^ ya));
        carry.b = (xb & yb) | (carry.b & (xb ^ yb));
    }
#pragma unroll
    for (int b = 7; b < kBits; ++b) {
        const uint64_t xa = acc[b].a, xb = acc[b].b;
        acc[b].a = xa ^ carry.a;
        acc[b].b = xb ^ carry.b;
        carry.a &= xa;
        carry.b &= xb;
    }
}

// One term decoded from its expressions (rows whose program found no slice).
template <bool kBuf>
__device__ Words pref_term_decoded(const pc_pred *__restrict__ preds, int64_t b, int64_t e,
                                   const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
                                   const Planes<kBuf> &pl)
{
    Words a{~0ull, ~0ull};
    for (int64_t p = b; p < e; ++p) {
        const pc_pred q = preds[p];
        const uint64_t *pres = present + static_cast<int64_t>(q.label) * 4;
        const uint32_t *wb = wbase + static_cast<int64_t>(q.label) * 4;
        uint64_t sel[4];
        bool neg;
        expr_clause(q.op, q.vals, pres, sel, neg);
        Words c{0, 0};
        for (int k = 0; k < 4; ++k) {
            uint64_t m = sel[k];
            while (m) {
                const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
                m &= m - 1;
                const Words x = pl(plane_id(pres, wb, v));
                c.a |= x.a;
                c.b |= x.b;
            }
        }
        a.a &= neg ? ~c.a : c.a;
        a.b &= neg ? ~c.b : c.b;
    }
    return a;
}

// Work item (tile of 128 words, chunk of rows) as in k_sel_eval; one row at
// a time per wavefront.  Per row: the feasible words (every node when the
// bitset is absent), the bit-sliced scores of the live terms, the lane's
// best (score, lowest node) and tie count, reduced over the wavefront into
// part_key[tile * I + r] = (score + 1) << 32 | ~node (0: no feasible node)
// and part_cnt[tile * I + r].
// kCls: the rows of one class list (0: scores within 8 bits, 1: within 16
// bits, 2: decoded on the fly, 3: at most three live terms), so that each
// launch keeps only the score words it needs and the common one carries no
// decoding code.  Class 3 keeps the (at most) three term masks instead of
// score bits: a node's score is fixed by the pattern of terms that hold for
// it, so the lane's best score is the largest pattern score whose node
// set meets its candidates, and its best nodes are the union of the
// candidates in the patterns of that score.
template <bool kBuf, int kCls>
__global__ __launch_bounds__(kEvalThreads) void k_pref_eval(
    const uint32_t *__restrict__ rec, const uint32_t *__restrict__ prog, const int32_t *__restrict__ row_off,
    const int32_t *__restrict__ term_off, const uint32_t *__restrict__ weight, const pc_pred *__restrict__ preds,
    int64_t n_preds, int32_t L, const uint64_t *__restrict__ present, const uint32_t *__restrict__ wbase,
    const uint64_t *__restrict__ planes, int64_t plane_bytes, int64_t Wp, int32_t I, int32_t W, int32_t N,
    const uint64_t *__restrict__ feasible, uint64_t *__restrict__ part_key, uint32_t *__restrict__ part_cnt,
    int32_t ntiles, int32_t nchunks, int32_t rpc, const int32_t *__restrict__ list,
    const uint32_t *__restrict__ list_len, int64_t fstride)
{
    constexpr int kBits = kCls == 0 ? 8 : (kCls == 3 ? 1 : kScoreBits);
    constexpr bool kDecode = kCls == 2;
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
    Planes<kBuf> pl;
    if constexpr (kBuf)
        pl.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(planes), static_cast<short>(0),
                                                    static_cast<int>(plane_bytes), 0x00020000);
    pl.lane_off = static_cast<uint32_t>(kPad + w0) * 8u;  // inside the plane row: kPad + w0 + 1 < Wp
    pl.rowbytes = static_cast<uint32_t>(Wp * 8);
    pl.pcol = planes + kPad + w0;
    pl.Wp = Wp;
    const int32_t *rows = list + static_cast<int64_t>(kCls) * I;
    const int32_t r0 = chunk * rpc;
    const int32_t r1 = min(static_cast<int32_t>(list_len[kCls]), r0 + rpc);
    // class 3: each wavefront stages its 64-row batch's records in LDS
    // (one record per lane), so a row's program words cost an LDS read
    // instead of a dependent memory load
    __shared__ uint4 lrec_all[kCls == 3 ? kEvalThreads * (kPrefRec / 4) : 1];
    const uint32_t *lrec = reinterpret_cast<const uint32_t *>(lrec_all + (kCls == 3 ? wave * 64 * (kPrefRec / 4) : 0));
    for (int32_t bat = r0 + wave * 64; bat < r1; bat += kEvalThreads) {
        const int32_t nb_rows = min(64, r1 - bat);
        // The batch's row ids, one per lane.  A row's record head and
        // feasible words (fstride 0: one all-ones row; lanes past the row's
        // end read its word 0 and mask it) are requested at the end of the
        // previous row, so their latency hides behind that row's selection.
        const int32_t my_row = lane < nb_rows ? rows[bat + lane] : 0;
        if constexpr (kCls == 3) {
            // the previous batch's reads are done (LDS requests of one
            // wavefront complete in order; the fences keep the compiler's
            // order)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            if (lane < nb_rows) {
                const uint4 *src = reinterpret_cast<const uint4 *>(rec + static_cast<int64_t>(my_row) * kPrefRec);
                uint4 *dst = lrec_all + (wave * 64 + lane) * (kPrefRec / 4);
#pragma unroll
                for (int q = 0; q < kPrefRec / 4; ++q) dst[q] = src[q];
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        auto feas_words = [&](int32_t rr, uint64_t &a, uint64_t &b) {
            const uint64_t *fr = feasible + static_cast<int64_t>(rr) * fstride;
            a = fr[ok0 ? w0 : 0];
            b = fr[ok1 ? w0 + 1 : 0];
        };
        int32_t r_next = __builtin_amdgcn_readlane(my_row, 0);
        uint32_t head_next = rec[static_cast<int64_t>(r_next) * kPrefRec];
        uint64_t fa_next, fb_next;
        feas_words(r_next, fa_next, fb_next);
        for (int32_t i = 0; i < nb_rows; ++i) {
            const int32_t r = r_next;
            const uint32_t *R = rec + static_cast<int64_t>(r) * kPrefRec;
            const uint32_t head = kCls == 3 ? lrec[i * kPrefRec] : head_next;
            const uint32_t kind = head >> 24, live = head & 0xFFFFu;
            const uint64_t fa = fa_next, fb = fb_next;
            Words cand{m0 & fa, m1 & fb};
            uint32_t sc = 0;
            if constexpr (kCls == 3) {
                Words A[kPrefFewTerms];
                uint32_t wt[kPrefFewTerms];
                const uint32_t nt = kind == kPrefNone ? 0u : live;
#pragma unroll
                for (int t = 0; t < static_cast<int>(kPrefFewTerms); ++t) {
                    A[t] = Words{0, 0};
                    wt[t] = 0;
                }
                // the program: inline words from the LDS copy, or a slice of
                // prog; one walk for either source, inlined at each call
                auto walk = [&](const uint32_t *pr) {
#pragma unroll
                for (int t = 0; t < static_cast<int>(kPrefFewTerms); ++t) {
                    if (static_cast<uint32_t>(t) < nt) {
                        const uint32_t hdr = *pr++;
                        wt[t] = hdr >> kPrefLenBits;
                        const int32_t len = static_cast<int32_t>(hdr & ((1u << kPrefLenBits) - 1));
                        Words a{~0ull, ~0ull}, c{0, 0}, unused{0, 0};
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
                                if (e0 + k < len) fold<false>(E[k], V[k], c, a, unused);
                        }
                        pr += len;
                        A[t] = a;
                    }
                }
                };
                if (kind == kPrefInline)
                    walk(lrec + i * kPrefRec + 2);
                else if (kind == kPrefIndirect)
                    walk(prog + lrec[i * kPrefRec + 1]);
                // pattern p: term t holds iff bit t of p (terms past nt hold
                // nowhere, so only p < 2^nt has nodes)
                auto pattern = [&](int p) {
                    Words m{~0ull, ~0ull};
#pragma unroll
                    for (int t = 0; t < static_cast<int>(kPrefFewTerms); ++t) {
                        m.a &= ((p >> t) & 1) ? A[t].a : ~A[t].a;
                        m.b &= ((p >> t) & 1) ? A[t].b : ~A[t].b;
                    }
                    return Words{m.a & cand.a, m.b & cand.b};
                };
                bool found = false;
#pragma unroll
                for (int p = 0; p < (1 << kPrefFewTerms); ++p) {
                    if (static_cast<uint32_t>(p) < (1u << nt)) {
                        const uint32_t sp = ((p & 1) ? wt[0] : 0u) + ((p & 2) ? wt[1] : 0u) + ((p & 4) ? wt[2] : 0u);
                        const Words t = pattern(p);
                        const bool any = (t.a | t.b) != 0;
                        sc = any && (!found || sp > sc) ? sp : sc;
                        found = found || any;
                    }
                }
                Words best{0, 0};
#pragma unroll
                for (int p = 0; p < (1 << kPrefFewTerms); ++p) {
                    if (static_cast<uint32_t>(p) < (1u << nt)) {
                        const uint32_t sp = ((p & 1) ? wt[0] : 0u) + ((p & 2) ? wt[1] : 0u) + ((p & 4) ? wt[2] : 0u);
                        const Words t = pattern(p);
                        const bool take = found && sp == sc;
                        best.a |= take ? t.a : 0ull;
                        best.b |= take ? t.b : 0ull;
                    }
                }
                cand = best;
            } else {
                Words acc[kBits];
#pragma unroll
                for (int b = 0; b < kBits; ++b) acc[b] = Words{0, 0};
                // one loop over the row's terms, whatever their source, so the
                // score words have a single update site
                constexpr bool dec = kDecode;
                const int64_t tb = dec ? row_off[r] : 0;
                const uint32_t n_iter = dec ? static_cast<uint32_t>(row_off[r + 1] - tb)
                                            : (kind == kPrefNone ? 0u : live);
                const uint32_t *pr = kind == kPrefInline ? R + 2 : prog + R[1];
                for (uint32_t t = 0; t < n_iter; ++t) {
                    uint32_t w;
                    Words a{~0ull, ~0ull};
                    if constexpr (dec) {
                        w = weight[tb + t];
                        int64_t len;
                        if (!pref_weight_ok(w) ||
                            !aff_term(preds, term_off[tb + t], term_off[tb + t + 1], n_preds, L, present, len))
                            continue;
                        a = pref_term_decoded<kBuf>(preds, term_off[tb + t], term_off[tb + t + 1], present, wbase, pl);
                    } else {
                        const uint32_t hdr = *pr++;
                        w = hdr >> kPrefLenBits;
                        const int32_t len = static_cast<int32_t>(hdr & ((1u << kPrefLenBits) - 1));
                        Words c{0, 0}, unused{0, 0};
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
                                if (e0 + k < len) fold<false>(E[k], V[k], c, a, unused);
                        }
                        pr += len;
                    }
                    score_add<kBits>(acc, w, a);
                }
                // best score among this lane's feasible nodes: keep the nodes
                // that have the highest remaining score bit set, top bit first
                auto narrow = [&](int b) {
                    const Words t{cand.a & acc[b].a, cand.b & acc[b].b};
                    const bool any = (t.a | t.b) != 0;
                    cand.a = any ? t.a : cand.a;
                    cand.b = any ? t.b : cand.b;
                    sc |= any ? (1u << b) : 0u;
                };
#pragma unroll
                for (int b = kBits - 1; b >= 0; --b) narrow(b);
            }
            if (i + 1 < nb_rows) {
                r_next = __builtin_amdgcn_readlane(my_row, i + 1);
                head_next = rec[static_cast<int64_t>(r_next) * kPrefRec];
                feas_words(r_next, fa_next, fb_next);
            }
            const bool has = (cand.a | cand.b) != 0;
            const uint32_t node = static_cast<uint32_t>(w0) * 64u +
                                  (cand.a ? static_cast<uint32_t>(__builtin_ctzll(cand.a))
                                          : 64u + static_cast<uint32_t>(__builtin_ctzll(cand.b | (1ull << 63))));
            // the wavefront's best score (+1; 0 = no feasible node), its
            // lowest node and the tie count
            const uint32_t top = wave_max_u32(has ? sc + 1 : 0u);
            const bool at_top = has && sc + 1 == top;
            const uint32_t nmin = wave_min_u32(at_top ? node : 0xFFFFFFFFu);
            const uint32_t cnt = wave_add_u32(at_top ? static_cast<uint32_t>(__popcll(cand.a) + __popcll(cand.b)) : 0u);
            const uint64_t key = top ? (static_cast<uint64_t>(top) << 32) | (0xFFFFFFFFu - nmin) : 0ull;
            if (lane == 0) {
                part_key[static_cast<int64_t>(tile) * I + r] = key;
                part_cnt[static_cast<int64_t>(tile) * I + r] = cnt;
            }
        }
    }
}

// Per row: the best key over the tiles and the tie count of that score.
__global__ __launch_bounds__(256) void k_pref_final(const uint64_t *__restrict__ part_key,
                                                    const uint32_t *__restrict__ part_cnt, int32_t I, int32_t ntiles,
                                                    int32_t *__restrict__ best, uint32_t *__restrict__ score,
                                                    uint32_t *__restrict__ count)
{
    const int32_t r = blockIdx.x * 256 + threadIdx.x;
    if (r >= I) return;
    uint64_t key = 0;
    for (int32_t t = 0; t < ntiles; ++t) {
        const uint64_t k = part_key[static_cast<int64_t>(t) * I + r];
        key = k > key ? k : key;
    }
    uint32_t cnt = 0;
    if (key != 0)
        for (int32_t t = 0; t < ntiles; ++t)
            if ((part_key[static_cast<int64_t>(t) * I + r] >> 32) == (key >> 32)) cnt += part_cnt[static_cast<int64_t>(t) * I + r];
    best[r] = key ? static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(key)) : -1;
    score[r] = key ? static_cast<uint32_t>(key >> 32) - 1u : 0u;
    count[r] = cnt;
}

}  // namespace

namespace {

// Evaluator geometry for N nodes: W bitset words per row, tiles of kTileW
// words, plane row pitch Wp.  Rows are shifted onto 128-byte lines when
// that costs no extra tile (W of at least one tile); every lane's word
// pair, shifted or not, lies inside [0, Wp - kPad) of a plane row.
struct EvalGeom {
    int64_t W, Wp, ntiles;
    int32_t shift;
};

EvalGeom eval_geom(int32_t N)
{
    EvalGeom g;
    g.W = (static_cast<int64_t>(N) + 63) / 64;
    g.ntiles = (g.W + kTileW - 1) / kTileW;
    g.shift = g.W >= kTileW && (g.W + 15 + kTileW - 1) / kTileW == g.ntiles;
    g.Wp = kPad + g.ntiles * kTileW;
    return g;
}

// Prefix planes of the affinity paths: plane pfx0 + plane_id(v) = OR of the
// planes of the label's present values <= v (v in 0..254), so that Gt / Lt
// take at most two entries (cmp_clause).  One thread per (label, plane
// word), over the label's present values in increasing order.
__global__ __launch_bounds__(256) void k_aff_prefix(const uint64_t *__restrict__ present,
                                                    const uint32_t *__restrict__ wbase, int32_t L,
                                                    uint64_t *__restrict__ planes, int64_t Wp, uint32_t pfx0)
{
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= static_cast<int64_t>(L) * Wp) return;
    const int32_t l = static_cast<int32_t>(idx / Wp);
    const int64_t w = idx % Wp;
    const uint64_t *pres = present + static_cast<int64_t>(l) * 4;
    const uint32_t *wb = wbase + static_cast<int64_t>(l) * 4;
    uint64_t acc = 0;
    for (int k = 0; k < 4; ++k) {
        uint64_t m = pres[k];
        if (k == 3) m &= ~(1ull << 63);  // the absent value has no prefix plane
        while (m) {
            const uint32_t v = static_cast<uint32_t>(k * 64 + __builtin_ctzll(m));
            m &= m - 1;
            const uint32_t pid = plane_id(pres, wb, v);
            acc |= planes[static_cast<int64_t>(pid) * Wp + w];
            planes[static_cast<int64_t>(pfx0 + pid) * Wp + w] = acc;
        }
    }
}

// Value planes of the node labels: presence, plane numbering (d_P = P),
// the planes themselves, and the all-zero plane pmax.
int build_planes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, int64_t W, int64_t Wp, int64_t pmax,
                 uint64_t *present, uint32_t *wbase, uint64_t *planes, int32_t *d_P, hipStream_t stream)
{
    launch_fill_u64(present, static_cast<size_t>(L) * 4, 0, stream);
    if (Wp > 0) launch_fill_u64(planes + static_cast<size_t>(pmax) * Wp, static_cast<size_t>(Wp), 0, stream);
    if (L == 0) launch_fill_u32(reinterpret_cast<uint32_t *>(d_P), 1, 0, stream);
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
    return PC_OK;
}

// The prefix planes pmax + 1 + [0, pmax) of the affinity paths (after
// build_planes).
int build_prefix(pc_ctx *ctx, int32_t L, int64_t Wp, int64_t pmax, const uint64_t *present, const uint32_t *wbase,
                 uint64_t *planes, hipStream_t stream)
{
    const int64_t n = static_cast<int64_t>(L) * Wp;
    if (n == 0) return PC_OK;
    PC_TIMED(ctx, "k_aff_prefix", stream,
             hipLaunchKernelGGL(k_aff_prefix, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream,
                                present, wbase, L, planes, Wp, static_cast<uint32_t>(pmax + 1)));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

// The evaluator over every row (feasible nullptr: popcounts only), then
// the popcount partials' sum.
template <bool kTerms>
int launch_eval(pc_ctx *ctx, const uint32_t *rec, const uint32_t *prog, const int32_t *off,
                const pc_pred *preds, const uint64_t *present, const uint32_t *wbase, const uint64_t *planes,
                int64_t pmax, int64_t Wp, int32_t I, int64_t W, int32_t N, uint64_t *feasible, uint32_t *popcnt,
                uint32_t *part, int64_t ntiles, const int32_t *term_off, int64_t n_preds, int32_t L,
                int32_t shift, hipStream_t stream)
{
    // about 32,768 workgroups (many per workgroup slot of the chip, so the
    // last wave of workgroups is short); a chunk is a whole number of
    // 64-row batches
    int64_t nchunks = std::max<int64_t>((32768 + ntiles - 1) / ntiles, 1);
    int64_t rpc = (I + nchunks - 1) / nchunks;
    rpc = (rpc + 63) / 64 * 64;
    nchunks = (I + rpc - 1) / rpc;
    const int64_t total = ntiles * nchunks;
    const unsigned blocks = static_cast<unsigned>(8 * ((total + 7) / 8));
    uint32_t *cnt_out = ntiles > 1 ? part : popcnt;
    const int64_t pbytes = static_cast<int64_t>(pmax + 1) * Wp * 8;
    auto eval = [&](auto kern) {
        PC_TIMED(ctx, kTerms ? "k_aff_eval" : (feasible ? "k_sel_eval" : "k_sel_count"), stream,
                 hipLaunchKernelGGL(kern, dim3(blocks), dim3(kEvalThreads), 0, stream, rec, prog, off, preds,
                                    present, wbase, planes, pbytes, Wp, I, static_cast<int32_t>(W), N, feasible,
                                    cnt_out, static_cast<int32_t>(ntiles), static_cast<int32_t>(nchunks),
                                    static_cast<int32_t>(rpc), term_off, n_preds, L, shift));
    };
    if (!feasible) {
        if (pbytes < (int64_t(1) << 31)) eval(k_sel_eval<true, kTerms, false>);  // buffer offsets are 32-bit
        else eval(k_sel_eval<false, kTerms, false>);
    } else {
        if (pbytes < (int64_t(1) << 31)) eval(k_sel_eval<true, kTerms>);
        else eval(k_sel_eval<false, kTerms>);
    }
    PC_LAUNCH_CHECK(ctx);
    if (ntiles > 1) {
        PC_TIMED(ctx, kTerms ? "k_aff_popsum" : "k_sel_popsum", stream,
                 hipLaunchKernelGGL(k_sel_popsum, dim3(static_cast<unsigned>((I + 255) / 256)), dim3(256), 0, stream,
                                    part, I, static_cast<int32_t>(ntiles), popcnt));
        PC_LAUNCH_CHECK(ctx);
    }
    return PC_OK;
}

}  // namespace

int run_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                  const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                  hipStream_t stream, char *fixed, size_t fixed_cap)
{
    const EvalGeom geo = eval_geom(N);
    const int64_t W = geo.W, Wp = geo.Wp, ntiles = geo.ntiles;
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
    char *base = fixed;
    if (fixed != nullptr) {
        if (dry.off > fixed_cap)
            return pc_set_error(ctx, PC_EINVAL,
                                "pc_eval_selectors_noalloc: needs %zu bytes of scratch, above its maximum of %zu "
                                "(N=%d L=%d I=%d n_preds=%lld)",
                                dry.off, fixed_cap, N, L, I, static_cast<long long>(n_preds));
    } else {
        int rc = pc_ensure_arena(ctx, dry.off);
        if (rc) return rc;
        base = ctx->arena;
    }
    Carver real{base, 0};
    carve(real);
    int rc = PC_OK;

    if (W == 0) launch_fill_u32(popcnt, static_cast<size_t>(I), 0, stream);
    rc = build_planes(ctx, labels, N, L, W, Wp, pmax, present, wbase, planes, d_P, stream);
    if (rc) return rc;
    const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>((I + 255) / 256, 8192));
    PC_TIMED(ctx, "k_sel_compile", stream,
             hipLaunchKernelGGL(k_sel_compile, dim3(rgrid), dim3(256), 0, stream, pred_off, preds, n_preds, I, L,
                                present, wbase, prog, rec, ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    if (W == 0) return PC_OK;
    return launch_eval<false>(ctx, rec, prog, pred_off, preds, present, wbase, planes, pmax, Wp, I, W, N, feasible,
                              popcnt, part, ntiles, nullptr, n_preds, L, geo.shift, stream);
}

int run_affinity(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *row_off, int32_t I,
                 const int32_t *term_off, int32_t n_terms, const pc_pred *preds, int64_t n_preds, uint64_t *feasible,
                 uint32_t *popcnt, uint8_t *unknown, hipStream_t stream)
{
    const EvalGeom geo = eval_geom(N);
    const int64_t W = geo.W, Wp = geo.Wp, ntiles = geo.ntiles;
    const int64_t pmax = static_cast<int64_t>(L) * (N < 256 ? N : 256);
    // value planes [0, pmax), the all-zero plane pmax, prefix planes pmax + 1 + [0, pmax)
    const int64_t ptop = 2 * pmax;
    const size_t plane_bytes = static_cast<size_t>(ptop + 1) * static_cast<size_t>(Wp) * 8;
    if (plane_bytes > (size_t(64) << 30))
        return pc_set_error(ctx, PC_ENOMEM, "pc_eval_affinity: value planes need %zu bytes (L=%d N=%d)", plane_bytes,
                            L, N);
    // indirect programs take slices of prog: room for 4 entries per
    // expression on average, rounded per row; the rest decode on the fly
    const int64_t prog_cap = 4 * n_preds + 4 * static_cast<int64_t>(I) + 64;
    uint64_t *present, *planes;
    uint32_t *wbase, *prog, *rec, *part;
    int32_t *d_P;
    unsigned long long *prog_used;
    auto carve = [&](Carver &cv) {
        present = cv.take<uint64_t>(static_cast<size_t>(L) * 4 + 1);
        wbase = cv.take<uint32_t>(static_cast<size_t>(L) * 4 + 1);
        planes = cv.take<uint64_t>(static_cast<size_t>(ptop + 1) * Wp + 2);
        prog = cv.take<uint32_t>(static_cast<size_t>(prog_cap));
        rec = cv.take<uint32_t>(static_cast<size_t>(I) * kRecWords + kRecWords);
        part = ntiles > 1 ? cv.take<uint32_t>(static_cast<size_t>(ntiles) * I + 1) : nullptr;
        d_P = cv.take<int32_t>(1);
        prog_used = cv.take<unsigned long long>(1);
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    const int64_t nval = std::max<int64_t>(I, n_terms);
    if (nval > 0) {
        const unsigned vgrid = static_cast<unsigned>(std::min<int64_t>((nval + 255) / 256, 8192));
        PC_TIMED(ctx, "k_aff_validate", stream,
                 hipLaunchKernelGGL(k_aff_validate, dim3(vgrid), dim3(256), 0, stream, row_off, I, term_off, n_terms,
                                    preds, n_preds, L, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (I == 0) return PC_OK;
    if (W == 0) launch_fill_u32(popcnt, static_cast<size_t>(I), 0, stream);
    launch_fill_u64(reinterpret_cast<uint64_t *>(prog_used), 1, 0, stream);
    rc = build_planes(ctx, labels, N, L, W, Wp, pmax, present, wbase, planes, d_P, stream);
    if (rc) return rc;
    rc = build_prefix(ctx, L, Wp, pmax, present, wbase, planes, stream);
    if (rc) return rc;
    const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>((I + 255) / 256, 8192));
    PC_TIMED(ctx, "k_aff_compile", stream,
             hipLaunchKernelGGL(k_aff_compile, dim3(rgrid), dim3(256), 0, stream, row_off, I, term_off, n_terms,
                                preds, n_preds, L, present, wbase, prog, prog_cap,
                                prog_used, rec, unknown, static_cast<uint32_t>(pmax + 1)));
    PC_LAUNCH_CHECK(ctx);
    if (W == 0) return PC_OK;
    return launch_eval<true>(ctx, rec, prog, row_off, preds, present, wbase, planes, ptop, Wp, I, W, N, feasible,
                             popcnt, part, ntiles, term_off, n_preds, L, geo.shift, stream);
}

int run_preferred(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const uint64_t *feasible,
                  const int32_t *row_off, int32_t I, const int32_t *term_off, int32_t n_terms, const uint32_t *weight,
                  const pc_pred *preds, int64_t n_preds, int32_t *best, uint32_t *score, uint32_t *count,
                  hipStream_t stream)
{
    const int64_t W = (static_cast<int64_t>(N) + 63) / 64;
    const int64_t ntiles = (W + kTileW - 1) / kTileW;
    const int64_t Wp = kPad + ntiles * kTileW;  // unshifted tiles: every lane's pair lies inside a plane row
    const int64_t pmax = static_cast<int64_t>(L) * (N < 256 ? N : 256);
    const int64_t ptop = 2 * pmax;  // value planes, the all-zero plane pmax, prefix planes
    const size_t plane_bytes = static_cast<size_t>(ptop + 1) * static_cast<size_t>(Wp) * 8;
    if (plane_bytes > (size_t(64) << 30))
        return pc_set_error(ctx, PC_ENOMEM, "pc_score_preferred: value planes need %zu bytes (L=%d N=%d)",
                            plane_bytes, L, N);
    // room for a header per term and 4 entries per expression; rows beyond it decode on the fly
    const int64_t prog_cap = std::min<int64_t>(static_cast<int64_t>(n_terms) + 4 * n_preds + 64, int64_t(1) << 31);
    uint64_t *present, *planes, *part_key, *ones;
    uint32_t *wbase, *prog, *rec, *part_cnt, *list_len;
    int32_t *d_P, *list;
    unsigned long long *prog_used;
    auto carve = [&](Carver &cv) {
        present = cv.take<uint64_t>(static_cast<size_t>(L) * 4 + 1);
        wbase = cv.take<uint32_t>(static_cast<size_t>(L) * 4 + 1);
        planes = cv.take<uint64_t>(static_cast<size_t>(ptop + 1) * Wp + 2);
        prog = cv.take<uint32_t>(static_cast<size_t>(prog_cap));
        rec = cv.take<uint32_t>(static_cast<size_t>(I) * kPrefRec + kPrefRec);
        list = cv.take<int32_t>(static_cast<size_t>(I) * kPrefClasses + 1);
        list_len = cv.take<uint32_t>(kPrefClasses);
        ones = cv.take<uint64_t>(feasible ? 1 : static_cast<size_t>(W) + 1);
        part_key = cv.take<uint64_t>(static_cast<size_t>(ntiles) * I + 1);
        part_cnt = cv.take<uint32_t>(static_cast<size_t>(ntiles) * I + 1);
        d_P = cv.take<int32_t>(1);
        prog_used = cv.take<unsigned long long>(1);
    };
    Carver dry{nullptr, 0};
    carve(dry);
    int rc = pc_ensure_arena(ctx, dry.off);
    if (rc) return rc;
    Carver real{ctx->arena, 0};
    carve(real);

    const int64_t nval = std::max<int64_t>(I, n_terms);
    if (nval > 0) {
        const unsigned vgrid = static_cast<unsigned>(std::min<int64_t>((nval + 255) / 256, 8192));
        PC_TIMED(ctx, "k_pref_validate", stream,
                 hipLaunchKernelGGL(k_pref_validate, dim3(vgrid), dim3(256), 0, stream, row_off, I, term_off, n_terms,
                                    weight, preds, n_preds, L, ctx->d_err));
        PC_LAUNCH_CHECK(ctx);
    }
    if (I == 0) return PC_OK;
    launch_fill_u64(reinterpret_cast<uint64_t *>(prog_used), 1, 0, stream);
    launch_fill_u32(list_len, kPrefClasses, 0, stream);
    if (!feasible && W > 0) launch_fill_u64(ones, static_cast<size_t>(W), ~0ull, stream);
    rc = build_planes(ctx, labels, N, L, W, Wp, pmax, present, wbase, planes, d_P, stream);
    if (rc) return rc;
    rc = build_prefix(ctx, L, Wp, pmax, present, wbase, planes, stream);
    if (rc) return rc;
    const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>((I + 255) / 256, 8192));
    PC_TIMED(ctx, "k_pref_compile", stream,
             hipLaunchKernelGGL(k_pref_compile, dim3(rgrid), dim3(256), 0, stream, row_off, I, term_off, n_terms,
                                weight, preds, n_preds, L, present, wbase, prog, prog_cap, prog_used, rec, list,
                                list_len, static_cast<uint32_t>(pmax + 1)));
    PC_LAUNCH_CHECK(ctx);
    if (W > 0) {
        int64_t nchunks = std::max<int64_t>((32768 + ntiles - 1) / ntiles, 1);
        int64_t rpc = (I + nchunks - 1) / nchunks;
        rpc = (rpc + 63) / 64 * 64;
        nchunks = (I + rpc - 1) / rpc;
        const int64_t total = ntiles * nchunks;
        const unsigned blocks = static_cast<unsigned>(8 * ((total + 7) / 8));
        const int64_t pbytes = static_cast<int64_t>(ptop + 1) * Wp * 8;
        auto eval = [&](auto kern, const char *name) {
            PC_TIMED(ctx, name, stream,
                     hipLaunchKernelGGL(kern, dim3(blocks), dim3(kEvalThreads), 0, stream, rec, prog, row_off, term_off,
                                        weight, preds, n_preds, L, present, wbase, planes, pbytes, Wp, I,
                                        static_cast<int32_t>(W), N, feasible ? feasible : ones, part_key, part_cnt,
                                        static_cast<int32_t>(ntiles), static_cast<int32_t>(nchunks),
                                        static_cast<int32_t>(rpc), list, list_len,
                                        feasible ? static_cast<int64_t>(W) : int64_t(0)));
        };
        // one launch per class list (sized for I rows; items past a list's
        // length exit at once)
        if (pbytes < (int64_t(1) << 31)) {
            eval(k_pref_eval<true, 0>, "k_pref_eval");
            eval(k_pref_eval<true, 1>, "k_pref_eval16");
            eval(k_pref_eval<true, 2>, "k_pref_decode");
            eval(k_pref_eval<true, 3>, "k_pref_eval3");
        } else {
            eval(k_pref_eval<false, 0>, "k_pref_eval");
            eval(k_pref_eval<false, 1>, "k_pref_eval16");
            eval(k_pref_eval<false, 2>, "k_pref_decode");
            eval(k_pref_eval<false, 3>, "k_pref_eval3");
        }
        PC_LAUNCH_CHECK(ctx);
    }
    PC_TIMED(ctx, "k_pref_final", stream,
             hipLaunchKernelGGL(k_pref_final, dim3(static_cast<unsigned>((I + 255) / 256)), dim3(256), 0, stream,
                                part_key, part_cnt, I, static_cast<int32_t>(W > 0 ? ntiles : 0), best, score, count));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}

// ---------------------------------------------------------------- fixed scratch
// The allocation-free selector entry point carves its scratch from this
// array instead of the context's arena.  Each device holds its own copy (the
// code object's memory, from the first use on that device until the process
// ends).  In host code the name stands for no device address: only the
// pointer hipGetSymbolAddress returns for the current device is used.  A
// 64 KiB guard band follows the usable PC_NOALLOC_SCRATCH_BYTES.
static __device__ __align__(256) unsigned char scratch[PC_NOALLOC_SCRATCH_BYTES + 65536];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices];  // this device's address of `scratch`, once looked up
}  // namespace

int pc_noalloc_setup(pc_ctx *ctx)
{
    if (ctx->device < 0 || ctx->device >= kMaxDevices)
        return pc_set_error(ctx, PC_EDEVICE, "device %d beyond the %d devices with fixed scratch", ctx->device,
                            kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[ctx->device] != nullptr) return PC_OK;
    void *p = nullptr;
    PC_HIP(ctx, hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return pc_set_error(ctx, PC_EDEVICE, "no device address for the fixed scratch");
    g_scratch_ptr[ctx->device] = static_cast<char *>(p);
    return PC_OK;
}

int run_selectors_noalloc(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                          const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                          hipStream_t stream)
{
    char *p = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (ctx->device >= 0 && ctx->device < kMaxDevices) p = g_scratch_ptr[ctx->device];
    }
    if (p == nullptr) return pc_set_error(ctx, PC_EDEVICE, "pc_eval_selectors_noalloc: fixed scratch not set up");
    return run_selectors(ctx, labels, N, L, pred_off, preds, n_preds, I, feasible, popcnt, stream, p,
                         PC_NOALLOC_SCRATCH_BYTES);
}

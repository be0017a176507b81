/*
 * Reference oracle for the cross-layer compliance check.  TEST
 * INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
 * baseline call it; the product path never does.
 *
 * Plain, slow, obviously correct scalar loops, parallelised only over the
 * outermost independent loop (rows, traces, queries).  It shares no code,
 * header or table with the GPU library; the record layouts below are
 * restated from the C ABI contract.
 *
 * What is computed (paper, Sec. "Formal Model and Satisfaction"): a
 * configuration satisfies an intent when (i) every placement constraint
 * holds for the nodes given their labels and (ii) every routing constraint
 * holds on the paths the installed flow rules realise; a validator check
 * is one atomic pass/fail assertion and an intent passes only when all of
 * its checks pass (Sec. "Automated Validation Pipeline", validator check
 * definition).
 *
 * Readings where the paper is silent (operator semantics, priority order,
 * ties, table miss, TTL, port model) are the ones listed with the C ABI:
 * Kubernetes node-affinity operators, larger priority wins, lower rule
 * index breaks ties, a table miss ends the trace, hops count links.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct { uint16_t label; uint8_t op; uint8_t rsv0; uint32_t rsv1; uint64_t vals[4]; } o_pred;
typedef struct { uint32_t value[4]; uint32_t mask[4]; uint16_t priority; uint16_t action; uint32_t rsv; } o_rule;
typedef struct { uint32_t jmask; int32_t last_switch; uint16_t last_port; uint8_t hops; uint8_t state; } o_trace;
typedef struct {
    uint8_t kind; uint8_t pad[3]; int32_t sel_row, src_node, dst_node, trace_begin, trace_end;
    uint32_t allowed; uint32_t pad2;
} o_intent;
typedef struct { int32_t dst_switch, dst_port, reach_q; } o_expect;
typedef struct { uint32_t must, forbid; } o_path_expect;
typedef struct { uint64_t counts[4][16]; uint64_t no_path[4]; } o_summary;

_Static_assert(sizeof(o_pred) == 40, "pred");
_Static_assert(sizeof(o_rule) == 40, "rule");
_Static_assert(sizeof(o_trace) == 12, "trace");
_Static_assert(sizeof(o_intent) == 32, "intent");
_Static_assert(sizeof(o_expect) == 12, "expect");
_Static_assert(sizeof(o_path_expect) == 8, "path expect");

enum { O_IN = 0, O_NOTIN = 1, O_EXISTS = 2 };
enum { O_EGRESS = 0, O_DROP = 1, O_MISS = 2, O_TTL = 3 };
/* data-error flags (sticky word).  A flag is raised when ANY item of the
 * corresponding input array is malformed, whichever rows, traces or queries
 * are evaluated; the evaluation itself gives malformed items a neutral
 * meaning and never reads out of bounds. */
enum { F_PRED = 1, F_OFFSETS = 2, F_ACTION = 4, F_SWITCH = 8, F_JUR = 16, F_GRAPH = 32, F_INTENT = 64, F_NODE = 128 };

static void set_flag(uint32_t *err, uint32_t f)
{
#pragma omp atomic
    *err |= f;
}

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------ A1
 * Selector rows (paper: a placement constraint such as a residency region
 * the chosen node must carry as a label, compiled to a Kubernetes node
 * selector / affinity; Formal Model and Satisfaction).  A row is a conjunction of predicates; a predicate
 * names one label and an operator:
 *   In S     : the node has the label and its value is in S
 *   NotIn S  : the node lacks the label, or its value is not in S
 *   Exists   : the node has the label
 * Label value 0xFF means "absent".  Output bit n of row r is set iff node n
 * satisfies every predicate of row r; words are LSB-first, W = ceil(N/64),
 * padding bits zero.  An empty row holds for every node.  A malformed
 * predicate (label >= L, op > 2, reserved field set, or value 255 in an
 * In/NotIn set) holds for no node (F_PRED); a malformed offset pair makes
 * the whole row empty (F_OFFSETS).
 */
static int pred_valid(const o_pred *q, int64_t L)
{
    return q->label < L && q->op <= 2 && q->rsv0 == 0 && q->rsv1 == 0 &&
           (q->op == O_EXISTS || ((q->vals[3] >> 63) & 1) == 0);
}

static int range_ok(int64_t b, int64_t e, int64_t n)
{
    return b >= 0 && e >= b && e <= n;
}

void orc_selectors(const uint8_t *labels, int64_t N, int64_t L,
                   const int32_t *pred_off, const o_pred *preds, int64_t n_preds, int64_t I,
                   const int32_t *rows, int64_t nrows,
                   uint64_t *feasible, uint32_t *popcnt, uint32_t *err, int nthreads)
{
    const int64_t W = (N + 63) / 64;
    set_threads(nthreads);
    /* data-error flags are a property of the inputs, independent of which rows are evaluated:
     * a malformed offset pair, or a malformed predicate inside a well-formed row */
    for (int64_t i = 0; i < I; ++i) {
        if (!range_ok(pred_off[i], pred_off[i + 1], n_preds)) { *err |= F_OFFSETS; continue; }
        for (int64_t p = pred_off[i]; p < pred_off[i + 1]; ++p)
            if (!pred_valid(&preds[p], L)) *err |= F_PRED;
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows[r];
        uint64_t *out = feasible + r * W;
        for (int64_t w = 0; w < W; ++w) out[w] = 0;
        uint32_t count = 0;
        const int64_t b = pred_off[i], e = pred_off[i + 1];
        if (!range_ok(b, e, n_preds)) {
            popcnt[r] = 0;
            continue;
        }
        for (int64_t n = 0; n < N; ++n) {
            int ok = 1;
            for (int64_t p = b; p < e; ++p) {
                const o_pred *q = &preds[p];
                if (!pred_valid(q, L)) {
                    ok = 0;
                    continue;
                }
                const unsigned x = labels[n * L + q->label];
                const int present = x != 0xFF;
                const int in_set = present && ((q->vals[x >> 6] >> (x & 63)) & 1);
                int sat;
                if (q->op == O_IN) sat = in_set;
                else if (q->op == O_NOTIN) sat = !in_set;
                else sat = present;
                if (!sat) ok = 0;
            }
            if (ok) {
                out[n >> 6] |= (uint64_t)1 << (n & 63);
                ++count;
            }
        }
        popcnt[r] = count;
    }
}

/* ------------------------------------------------------------------ A1 (incremental)
 * Continuous re-validation after a label change (paper, Abstract: the
 * validator is meant for continuous cross-layer compliance checking; the
 * cluster state the placement checks read changes as nodes are relabelled).  The labels of the listed nodes have changed; every other
 * node's labels are as when feasible / popcnt were computed.  For every
 * row r and, in list order, every listed node n: the row's bit of n is set
 * to the selector definition on n's new labels, and popcnt[r] moves by the
 * change of that bit.  A listed node outside [0, N) is skipped (F_NODE).
 * Rows and predicates have the meaning and the flags of orc_selectors.
 */
static int row_holds(const uint8_t *lab, int64_t L, const o_pred *preds, int64_t b, int64_t e)
{
    for (int64_t p = b; p < e; ++p) {
        const o_pred *q = &preds[p];
        if (!pred_valid(q, L)) return 0;
        const unsigned x = lab[q->label];
        const int present = x != 0xFF;
        const int in_set = present && ((q->vals[x >> 6] >> (x & 63)) & 1);
        const int sat = q->op == O_IN ? in_set : q->op == O_NOTIN ? !in_set : present;
        if (!sat) return 0;
    }
    return 1;
}

void orc_update_nodes(const uint8_t *labels, int64_t N, int64_t L, const int32_t *pred_off, const o_pred *preds,
                      int64_t n_preds, int64_t I, const int32_t *nodes, int64_t M, uint64_t *feasible,
                      uint32_t *popcnt, uint32_t *err, int nthreads)
{
    const int64_t W = (N + 63) / 64;
    set_threads(nthreads);
    for (int64_t i = 0; i < I; ++i) {
        if (!range_ok(pred_off[i], pred_off[i + 1], n_preds)) { *err |= F_OFFSETS; continue; }
        for (int64_t p = pred_off[i]; p < pred_off[i + 1]; ++p)
            if (!pred_valid(&preds[p], L)) *err |= F_PRED;
    }
    for (int64_t m = 0; m < M; ++m)
        if (nodes[m] < 0 || nodes[m] >= N) *err |= F_NODE;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t r = 0; r < I; ++r) {
        const int64_t b = pred_off[r], e = pred_off[r + 1];
        const int ok_row = range_ok(b, e, n_preds);
        for (int64_t m = 0; m < M; ++m) {
            const int64_t n = nodes[m];
            if (n < 0 || n >= N) continue;
            const int now = ok_row && row_holds(labels + n * L, L, preds, b, e);
            uint64_t *w = &feasible[r * W + (n >> 6)];
            const uint64_t bit = (uint64_t)1 << (n & 63);
            const int was = (*w & bit) != 0;
            if (now && !was) { *w |= bit; popcnt[r] += 1; }
            if (!now && was) { *w &= ~bit; popcnt[r] -= 1; }
        }
    }
}

/* ------------------------------------------------------------------ A1 (probes)
 * Membership queries for verdict-only runs: bit[k] = whether node
 * probe_node[k] satisfies selector row probe_row[k] (the selector
 * definition above); 0 and F_NODE when the row or the node is out of range.
 * Rows and predicates have the meaning and the flags of orc_selectors.
 */
void orc_probes(const uint8_t *labels, int64_t N, int64_t L, const int32_t *pred_off, const o_pred *preds,
                int64_t n_preds, int64_t I, const int32_t *probe_row, const int32_t *probe_node, int64_t P,
                uint8_t *bit, uint32_t *err)
{
    for (int64_t i = 0; i < I; ++i) {
        if (!range_ok(pred_off[i], pred_off[i + 1], n_preds)) { *err |= F_OFFSETS; continue; }
        for (int64_t p = pred_off[i]; p < pred_off[i + 1]; ++p)
            if (!pred_valid(&preds[p], L)) *err |= F_PRED;
    }
    for (int64_t k = 0; k < P; ++k) {
        const int64_t r = probe_row[k], n = probe_node[k];
        bit[k] = 0;
        if (r < 0 || r >= I || n < 0 || n >= N) { *err |= F_NODE; continue; }
        const int64_t b = pred_off[r], e = pred_off[r + 1];
        bit[k] = (uint8_t)(range_ok(b, e, n_preds) && row_holds(labels + n * L, L, preds, b, e));
    }
}

/* ------------------------------------------------------------------ A1 (affinity)
 * Required node affinity (paper: placement directives become Kubernetes
 * node selection criteria and affinity rules, Sec. "Intent Translation",
 * "Service Placement Module"; the validator cross-checks every referenced
 * label against the live node-label inventory and fails a placement that
 * names a label no node carries, Sec. "Failure modes", hallucinated
 * identifiers).  Kubernetes semantics:
 *   a row holds for node n iff at least one of its terms holds; a term
 *   holds iff every one of its expressions holds.  A row with no terms
 *   holds for every node (no required affinity); a term with no
 *   expressions holds for no node.
 *   Operators: In, NotIn, Exists as for selector rows, and
 *     DoesNotExist : the node lacks the label
 *     Gt t / Lt t  : the node has the label and its value, read as the
 *                    integer it encodes (0..254), is > t / < t, where
 *                    t = (int64) vals[0].
 * Malformed: label >= L, op > 5, reserved field set, value 255 in an
 * In/NotIn set, or vals[1..3] != 0 for Gt/Lt -> the expression holds for
 * no node (F_PRED, raised for any such expression inside a well-formed
 * term); a bad term offset pair -> the term holds for no node, a bad row
 * offset pair -> the row holds for no node (F_OFFSETS, any pair).
 * Inventory flags per row (unknown[r]): bit 0 when a well-formed In/NotIn
 * expression of a well-formed term names a value no node carries for that
 * label; bit 1 when a well-formed expression names a label that every
 * node lacks.
 */
enum { O_DOESNOTEXIST = 3, O_GT = 4, O_LT = 5 };

static int aff_valid(const o_pred *q, int64_t L)
{
    if (q->label >= L || q->op > 5 || q->rsv0 != 0 || q->rsv1 != 0) return 0;
    if ((q->op == O_IN || q->op == O_NOTIN) && ((q->vals[3] >> 63) & 1)) return 0;
    if ((q->op == O_GT || q->op == O_LT) && (q->vals[1] | q->vals[2] | q->vals[3])) return 0;
    return 1;
}

static int aff_holds(const o_pred *q, unsigned x)
{
    const int present = x != 0xFF;
    const int in_set = present && ((q->vals[x >> 6] >> (x & 63)) & 1);
    const int64_t t = (int64_t)q->vals[0];
    switch (q->op) {
    case O_IN: return in_set;
    case O_NOTIN: return !in_set;
    case O_EXISTS: return present;
    case O_DOESNOTEXIST: return !present;
    case O_GT: return present && (int64_t)x > t;
    default: return present && (int64_t)x < t;  /* O_LT */
    }
}

void orc_affinity(const uint8_t *labels, int64_t N, int64_t L,
                  const int32_t *row_off, int64_t I, const int32_t *term_off, int64_t n_terms,
                  const o_pred *preds, int64_t n_preds, const int32_t *rows, int64_t nrows,
                  uint64_t *feasible, uint32_t *popcnt, uint8_t *unknown, uint32_t *err, int nthreads)
{
    const int64_t W = (N + 63) / 64;
    set_threads(nthreads);
    for (int64_t t = 0; t < n_terms; ++t) {
        if (!range_ok(term_off[t], term_off[t + 1], n_preds)) { *err |= F_OFFSETS; continue; }
        for (int64_t p = term_off[t]; p < term_off[t + 1]; ++p)
            if (!aff_valid(&preds[p], L)) *err |= F_PRED;
    }
    for (int64_t i = 0; i < I; ++i)
        if (!range_ok(row_off[i], row_off[i + 1], n_terms)) *err |= F_OFFSETS;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows[r];
        uint64_t *out = feasible + r * W;
        for (int64_t w = 0; w < W; ++w) out[w] = 0;
        popcnt[r] = 0;
        unknown[r] = 0;
        const int64_t tb = row_off[i], te = row_off[i + 1];
        if (!range_ok(tb, te, n_terms)) continue;
        /* inventory cross-check */
        for (int64_t t = tb; t < te; ++t) {
            if (!range_ok(term_off[t], term_off[t + 1], n_preds)) continue;
            for (int64_t p = term_off[t]; p < term_off[t + 1]; ++p) {
                const o_pred *q = &preds[p];
                if (!aff_valid(q, L)) continue;
                int key_seen = 0;
                for (int64_t n = 0; n < N && !key_seen; ++n) key_seen = labels[n * L + q->label] != 0xFF;
                if (!key_seen) unknown[r] |= 2;
                if (q->op == O_IN || q->op == O_NOTIN) {
                    for (unsigned v = 0; v < 255; ++v) {
                        if (!((q->vals[v >> 6] >> (v & 63)) & 1)) continue;
                        int seen = 0;
                        for (int64_t n = 0; n < N && !seen; ++n) seen = labels[n * L + q->label] == v;
                        if (!seen) unknown[r] |= 1;
                    }
                }
            }
        }
        uint32_t count = 0;
        for (int64_t n = 0; n < N; ++n) {
            int ok = te == tb;  /* no terms: no required affinity */
            for (int64_t t = tb; t < te && !ok; ++t) {
                const int64_t b = term_off[t], e = term_off[t + 1];
                if (!range_ok(b, e, n_preds) || b == e) continue;
                int tok = 1;
                for (int64_t p = b; p < e; ++p) {
                    const o_pred *q = &preds[p];
                    if (!aff_valid(q, L) || !aff_holds(q, labels[n * L + q->label])) tok = 0;
                }
                ok = tok;
            }
            if (ok) {
                out[n >> 6] |= (uint64_t)1 << (n & 63);
                ++count;
            }
        }
        popcnt[r] = count;
    }
}

/* ------------------------------------------------------------------ A1
 * Preferred node affinity: the secondary objective of placement (paper:
 * among the configurations that satisfy an intent, choose one that is
 * best for secondary objectives; Problem Definition, item 3), in the
 * Kubernetes form of weighted preferred terms (affinity rules of the
 * Placement Directives and the Service Placement Module).
 *   Row i owns the weighted terms row_off[i] .. row_off[i+1]; term t has
 *   weight weight[t] (1..100) and the expressions term_off[t] ..
 *   term_off[t+1], which hold as for required affinity (all of them must
 *   hold; a term without expressions holds for no node).
 *   score(i, n) = sum of the weights of row i's terms that hold for node n.
 *   Among the row's feasible nodes (bit n of feasible row i, or every node
 *   when feasible is NULL) the best node is the one of largest score, the
 *   lowest index among equal scores.  Reported per row: that node (-1 when
 *   no node is feasible), its score and the number of feasible nodes with
 *   that score (both 0 when no node is feasible).
 * Malformed: a weight outside 1..100 -> the term holds for no node
 * (F_PRED, any term); a malformed expression -> its term holds for no node
 * (F_PRED, as for required affinity); a bad term offset pair -> the term
 * holds for no node; a bad row offset pair or a row of more than
 * O_PREF_MAX_TERMS terms -> the row has no terms (F_OFFSETS, any row).
 */
enum { O_PREF_MAX_TERMS = 655 };

static int pref_row_ok(const int32_t *row_off, int64_t i, int64_t n_terms)
{
    return range_ok(row_off[i], row_off[i + 1], n_terms) && row_off[i + 1] - row_off[i] <= O_PREF_MAX_TERMS;
}

static int pref_term_holds(const uint8_t *lab, int64_t L, const int32_t *term_off, const uint32_t *weight,
                           const o_pred *preds, int64_t n_preds, int64_t t)
{
    const int64_t b = term_off[t], e = term_off[t + 1];
    if (weight[t] < 1 || weight[t] > 100 || !range_ok(b, e, n_preds) || b == e) return 0;
    for (int64_t p = b; p < e; ++p)
        if (!aff_valid(&preds[p], L) || !aff_holds(&preds[p], lab[preds[p].label])) return 0;
    return 1;
}

void orc_preferred(const uint8_t *labels, int64_t N, int64_t L, const uint64_t *feasible,
                   const int32_t *row_off, int64_t I, const int32_t *term_off, int64_t n_terms,
                   const uint32_t *weight, const o_pred *preds, int64_t n_preds, const int32_t *rows,
                   int64_t nrows, int32_t *best, uint32_t *score, uint32_t *count, uint32_t *err, int nthreads)
{
    const int64_t W = (N + 63) / 64;
    set_threads(nthreads);
    for (int64_t t = 0; t < n_terms; ++t) {
        if (weight[t] < 1 || weight[t] > 100) *err |= F_PRED;
        if (!range_ok(term_off[t], term_off[t + 1], n_preds)) { *err |= F_OFFSETS; continue; }
        for (int64_t p = term_off[t]; p < term_off[t + 1]; ++p)
            if (!aff_valid(&preds[p], L)) *err |= F_PRED;
    }
    for (int64_t i = 0; i < I; ++i)
        if (!pref_row_ok(row_off, i, n_terms)) *err |= F_OFFSETS;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows[r];
        const int ok = pref_row_ok(row_off, i, n_terms);
        const int64_t tb = ok ? row_off[i] : 0, te = ok ? row_off[i + 1] : 0;
        int64_t b_node = -1;
        uint32_t b_score = 0, b_count = 0;
        for (int64_t n = 0; n < N; ++n) {
            if (feasible && !((feasible[i * W + (n >> 6)] >> (n & 63)) & 1)) continue;
            uint32_t sc = 0;
            for (int64_t t = tb; t < te; ++t)
                if (pref_term_holds(labels + n * L, L, term_off, weight, preds, n_preds, t)) sc += weight[t];
            if (b_node < 0 || sc > b_score) {
                b_node = n;
                b_score = sc;
                b_count = 1;
            } else if (sc == b_score) {
                ++b_count;
            }
        }
        best[r] = (int32_t)b_node;
        score[r] = b_score;
        count[r] = b_count;
    }
}

/* ------------------------------------------------------------------ A3
 * Trace one header through the flow tables (paper: a routing constraint
 * is judged on the paths the installed rules actually realise, and flow
 * rules are compiled per hop along a path; Formal Model and Satisfaction,
 * Network orchestration).  At switch s the rule that
 * applies is the one of highest priority whose value agrees with the
 * header on every bit its mask cares about; equal priorities go to the
 * lower index within the switch's table.  No match: MISS.  Action 0xFFFF:
 * DROP.  Otherwise the action is a local port; a port with no peer switch
 * faces a host: EGRESS there.  A forward when `ttl` links have already been
 * crossed ends in TTL at the current switch.  jmask collects the
 * jurisdiction bit of every switch visited, the ingress included.
 * vsum (optional) summarises the visited switches for incremental
 * re-validation: bit (s mod 64) for every switch s on the walk, the
 * ingress included (0 for an invalid ingress).  walk (optional, 8 slots
 * per trace) holds the first 8 switches of the walk in order, -1 past its
 * end (all -1 for an invalid ingress).  A walk reads the tables of the
 * switches it visits only, so a walk that visits no changed switch is the
 * same walk after the change.
 */
static int rule_matches(const o_rule *r, const uint32_t *h)
{
    for (int w = 0; w < 4; ++w)
        if (((h[w] ^ r->value[w]) & r->mask[w]) != 0) return 0;
    return 1;
}

static uint32_t jur_bit(const uint8_t *jur, int64_t s)
{
    return jur[s] >= 32 ? 0 : (uint32_t)1 << jur[s];
}

void orc_trace(int64_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
               const uint8_t *jur, const int32_t *rule_off, const o_rule *rules, int64_t n_rules,
               const uint32_t *hdr, const int32_t *ingress, int64_t T, int64_t ttl,
               const int32_t *watch, int64_t K, const int64_t *idx, int64_t nidx, o_trace *out, uint32_t *visit,
               uint64_t *vsum, int32_t *walk, uint32_t *err, int nthreads)
{
    set_threads(nthreads);
    /* data-error flags: a sweep over every input item */
    for (int64_t t = 0; t < T; ++t)
        if (ingress[t] < 0 || ingress[t] >= S) { *err |= F_SWITCH; break; }
    for (int64_t i = 0; i < T * K; ++i)
        if (watch[i] < -1 || watch[i] >= S) { *err |= F_SWITCH; break; }
    for (int64_t p = 0; p < n_ports; ++p)
        if (port_peer[p] < -1 || port_peer[p] >= S) { *err |= F_SWITCH; break; }
    for (int64_t s = 0; s < S; ++s) {
        if (jur[s] >= 32) *err |= F_JUR;
        const int pok = range_ok(port_off[s], port_off[s + 1], n_ports);
        const int rok = range_ok(rule_off[s], rule_off[s + 1], n_rules);
        if (!pok || !rok) *err |= F_OFFSETS;
        if (!rok) continue;
        const int64_t np = pok ? port_off[s + 1] - port_off[s] : 0;
        for (int64_t r = rule_off[s]; r < rule_off[s + 1]; ++r)
            if (rules[r].action != 0xFFFF && (int64_t)rules[r].action >= np) { *err |= F_ACTION; break; }
    }
#pragma omp parallel
    {
    /* the switches the walk visits, in order (ingress first) */
    int64_t *path = (int64_t *)malloc(sizeof(int64_t) * (size_t)(ttl + 1));
#pragma omp for schedule(dynamic, 16)
    for (int64_t k = 0; k < nidx; ++k) {
        const int64_t t = idx[k];
        const uint32_t *h = hdr + 4 * t;
        o_trace res;
        int64_t s = ingress[t];
        res.last_port = 0xFFFF;
        res.hops = 0;
        if (visit) visit[k] = 0;
        if (vsum) vsum[k] = 0;
        if (walk)
            for (int j = 0; j < 8; ++j) walk[k * 8 + j] = -1;
        if (s < 0 || s >= S) {
            res.jmask = 0;
            res.last_switch = (int32_t)s;
            res.state = O_MISS;
            out[k] = res;
            continue;
        }
        uint32_t jm = jur_bit(jur, s);
        int64_t hops = 0;
        int64_t npath = 0;
        path[npath++] = s;
        int state;
        for (;;) {
            const int64_t rb = rule_off[s], re = rule_off[s + 1];
            int64_t best = -1;
            if (range_ok(rb, re, n_rules)) {
                for (int64_t r = rb; r < re; ++r) {
                    if (!rule_matches(&rules[r], h)) continue;
                    if (best < 0 || rules[r].priority > rules[best].priority) best = r;
                }
            }
            if (best < 0) { state = O_MISS; break; }
            const unsigned a = rules[best].action;
            if (a == 0xFFFF) { state = O_DROP; break; }
            const int64_t pb = port_off[s], pe = port_off[s + 1];
            if (!range_ok(pb, pe, n_ports) || (int64_t)a >= pe - pb) {
                state = O_MISS;
                break;
            }
            const int64_t peer = port_peer[pb + a];
            if (peer == -1) { state = O_EGRESS; res.last_port = (uint16_t)a; break; }
            if (peer < -1 || peer >= S) {
                state = O_MISS;
                break;
            }
            if (hops == ttl) { state = O_TTL; break; }
            s = peer;
            ++hops;
            jm |= jur_bit(jur, s);
            path[npath++] = s;
        }
        res.jmask = jm;
        res.last_switch = (int32_t)s;
        res.hops = (uint8_t)hops;
        res.state = (uint8_t)state;
        out[k] = res;
        /* watch slot j is set iff its switch is on the visited path (the
         * paper's must-go / forbidden checks over realised paths) */
        if (visit) {
            uint32_t m = 0;
            for (int64_t j = 0; j < K; ++j)
                for (int64_t p = 0; p < npath; ++p)
                    if (watch[t * K + j] == path[p]) { m |= (uint32_t)1 << j; break; }
            visit[k] = m;
        }
        if (vsum) {
            uint64_t m = 0;
            for (int64_t p = 0; p < npath; ++p) m |= (uint64_t)1 << (path[p] & 63);
            vsum[k] = m;
        }
        if (walk)
            for (int64_t p = 0; p < npath && p < 8; ++p) walk[k * 8 + p] = (int32_t)path[p];
    }
    free(path);
    }
}

/* ------------------------------------------------------------------ A5
 * Hop distance from src inside the subgraph induced by the allowed
 * switches: vertex v is allowed when bit region[v] of `allowed` is set
 * (region >= 32 is never allowed).  Textbook FIFO
 * breadth-first search over the undirected CSR graph.  A disallowed or
 * out-of-range source leaves every distance at -1.  With target == NULL
 * the full row [V] is written, else the single distance to target[q].
 */
void orc_reach(int64_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
               const uint8_t *region, int64_t Q, const int32_t *src, const uint32_t *allowed,
               const int32_t *target, const int64_t *qidx, int64_t nq,
               int32_t *dist_out, uint32_t *err, int nthreads)
{
    set_threads(nthreads);
    /* data-error flags: a sweep over every input item */
    for (int64_t v = 0; v < V; ++v) {
        if (region[v] >= 32) *err |= F_JUR;
        if (!range_ok(adj_off[v], adj_off[v + 1], n_adj)) *err |= F_OFFSETS;
    }
    for (int64_t p = 0; p < n_adj; ++p)
        if (adj[p] < 0 || adj[p] >= V) { *err |= F_GRAPH; break; }
    for (int64_t q = 0; q < Q; ++q) {
        if (src[q] < 0 || src[q] >= V) *err |= F_SWITCH;
        if (target && (target[q] < 0 || target[q] >= V)) *err |= F_SWITCH;
    }
#pragma omp parallel
    {
        int32_t *dist = (int32_t *)malloc(sizeof(int32_t) * (size_t)(V > 0 ? V : 1));
        int64_t *queue = (int64_t *)malloc(sizeof(int64_t) * (size_t)(V > 0 ? V : 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t k = 0; k < nq; ++k) {
            const int64_t q = qidx[k];
            for (int64_t v = 0; v < V; ++v) dist[v] = -1;
            const int64_t s = src[q];
            const uint32_t A = allowed[q];
            int64_t tgt = -1;
            int tgt_ok = 1;
            if (target) {
                tgt = target[q];
                if (tgt < 0 || tgt >= V) tgt_ok = 0;
            }
            int src_ok = 1;
            if (s < 0 || s >= V || region[s] >= 32 || !((A >> region[s]) & 1)) src_ok = 0;
            if (src_ok) {
                int64_t head = 0, tail = 0;
                dist[s] = 0;
                queue[tail++] = s;
                while (head < tail) {
                    const int64_t u = queue[head++];
                    const int64_t b = adj_off[u], e = adj_off[u + 1];
                    if (!range_ok(b, e, n_adj)) continue;
                    for (int64_t p = b; p < e; ++p) {
                        const int64_t v = adj[p];
                        if (v < 0 || v >= V) continue;
                        if (region[v] >= 32 || !((A >> region[v]) & 1)) continue;
                        if (dist[v] != -1) continue;
                        dist[v] = dist[u] + 1;
                        queue[tail++] = v;
                    }
                }
            }
            if (target) {
                dist_out[k] = tgt_ok ? dist[tgt] : -1;
            } else {
                memcpy(dist_out + k * V, dist, sizeof(int32_t) * (size_t)V);
            }
        }
        free(dist);
        free(queue);
    }
}

/* ------------------------------------------------------------------ A5, waypoints
 * Required waypoints and forbidden switches (paper: the routing constraints
 * of a Configuration name required waypoints and forbidden vertices; the
 * JSON constraints carry must_go and forbidden lists).  The walk must go
 * src -> via[0] -> ... -> via[m-1] -> target (m = entries before the first
 * -1) on switches that are allowed and not forbidden.  The shortest such
 * walk is the sum over its legs of the leg's shortest path, each found by a
 * textbook FIFO breadth-first search; a leg without a path makes the whole
 * distance -1.  Sums saturate at INT32_MAX.
 */
static int usable(const uint8_t *region, uint32_t A, const int32_t *fb, int64_t Kf, int64_t v)
{
    if (region[v] >= 32 || !((A >> region[v]) & 1)) return 0;
    for (int64_t k = 0; k < Kf; ++k)
        if (fb[k] == v) return 0;
    return 1;
}

static int64_t leg_bfs(int64_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                       const uint8_t *region, uint32_t A, const int32_t *fb, int64_t Kf, int64_t s, int64_t t,
                       int32_t *dist, int64_t *queue)
{
    if (s < 0 || s >= V || t < 0 || t >= V) return -1;
    if (!usable(region, A, fb, Kf, s)) return -1;
    for (int64_t v = 0; v < V; ++v) dist[v] = -1;
    int64_t head = 0, tail = 0;
    dist[s] = 0;
    queue[tail++] = s;
    while (head < tail) {
        const int64_t u = queue[head++];
        const int64_t b = adj_off[u], e = adj_off[u + 1];
        if (!range_ok(b, e, n_adj)) continue;
        for (int64_t p = b; p < e; ++p) {
            const int64_t v = adj[p];
            if (v < 0 || v >= V || dist[v] != -1) continue;
            if (!usable(region, A, fb, Kf, v)) continue;
            dist[v] = dist[u] + 1;
            queue[tail++] = v;
        }
    }
    return dist[t];
}

void orc_reach_via(int64_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                   const uint8_t *region, int64_t Q, const int32_t *src, const uint32_t *allowed,
                   const int32_t *target, const int32_t *via, int64_t Kv, const int32_t *forbid, int64_t Kf,
                   const int64_t *qidx, int64_t nq, int32_t *dist_out, uint32_t *err, int nthreads)
{
    set_threads(nthreads);
    for (int64_t v = 0; v < V; ++v) {
        if (region[v] >= 32) *err |= F_JUR;
        if (!range_ok(adj_off[v], adj_off[v + 1], n_adj)) *err |= F_OFFSETS;
    }
    for (int64_t p = 0; p < n_adj; ++p)
        if (adj[p] < 0 || adj[p] >= V) { *err |= F_GRAPH; break; }
    for (int64_t q = 0; q < Q; ++q)
        if (src[q] < 0 || src[q] >= V || target[q] < 0 || target[q] >= V) *err |= F_SWITCH;
    for (int64_t i = 0; i < Q * Kv; ++i)
        if (via[i] < -1 || via[i] >= V) { *err |= F_SWITCH; break; }
    for (int64_t i = 0; i < Q * Kf; ++i)
        if (forbid[i] < -1 || forbid[i] >= V) { *err |= F_SWITCH; break; }
#pragma omp parallel
    {
        int32_t *dist = (int32_t *)malloc(sizeof(int32_t) * (size_t)(V > 0 ? V : 1));
        int64_t *queue = (int64_t *)malloc(sizeof(int64_t) * (size_t)(V > 0 ? V : 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t k = 0; k < nq; ++k) {
            const int64_t q = qidx[k];
            const int32_t *w = via + q * Kv;
            const int32_t *fb = forbid + q * Kf;
            int64_t total = 0, from = src[q];
            int64_t m = 0;
            while (m < Kv && w[m] != -1) ++m;
            for (int64_t leg = 0; leg <= m; ++leg) {
                const int64_t to = leg < m ? w[leg] : target[q];
                const int64_t d = leg_bfs(V, adj_off, adj, n_adj, region, allowed[q], fb, Kf, from, to, dist, queue);
                if (d < 0) { total = -1; break; }
                total += d;
                from = to;
            }
            dist_out[k] = (int32_t)(total > 0x7FFFFFFF ? 0x7FFFFFFF : total);
        }
        free(dist);
        free(queue);
    }
}

/* ------------------------------------------------------------------ NEXT-2
 * Path synthesis (paper, Sec. "Network orchestration": a path scheduler
 * performs graph search over the current topology -- weighted Dijkstra,
 * BFS fallback -- to produce a path that respects the constraints, and
 * each path is turned into per-hop flow rules).
 * Graph: switch s owns ports port_off[s] .. port_off[s+1]; a port with
 * peer v in [0, V) and weight >= 1 is a link s -> v of that weight (weight
 * NULL: every link weighs 1, i.e. BFS).  A switch is usable by a request
 * when its region is allowed and it is not on the request's forbidden list.
 * Each leg (src -> via[0] -> ... -> target; the waypoint list ends at its
 * first -1) is a
 * minimum-weight path through usable switches; among those, the
 * predecessor of every switch v is the lowest-numbered u with a link
 * u -> v and dist(u) + w = dist(v) -- the lexicographically smallest path
 * read from its end.  The walk is the legs concatenated.  Switch path[k]
 * of the walk gets one rule: value = key, mask = the key's 104 bits,
 * priority = prio, action = its port of least (weight, index) to path[k+1],
 * or out_port at the last switch.
 * A request fails (hops -1, path -1, rules zero) when an endpoint or
 * waypoint is out of range, a leg has no path, out_port is not a port of
 * the target, or the walk has more than max_hops links.
 * Distances are sums of link weights below 2^31 - 1 (the paper gives no
 * range for them; this is the library's reading): a switch whose minimum
 * distance from the leg's start is 2^31 - 1 or more is unreachable, so a
 * leg whose target lies that far has no path.
 * Flags (input properties): OFFSETS bad port_off pair; SWITCH a peer < -1
 * or >= V, src / target outside [0, V), a via / forbid entry < -1 or >= V;
 * JUR region >= 32; GRAPH a zero weight (that port is no link); ACTION
 * out_port not a port of a target whose ports are well-formed.
 */
typedef struct { int64_t d; int64_t v; } ps_item;

#define PS_DIST_LIMIT ((int64_t)2147483647) /* distances stay below 2^31 - 1 */

static void heap_push(ps_item *h, int64_t *n, ps_item x)
{
    int64_t i = (*n)++;
    while (i > 0) {
        const int64_t par = (i - 1) / 2;
        if (h[par].d < x.d || (h[par].d == x.d && h[par].v <= x.v)) break;
        h[i] = h[par];
        i = par;
    }
    h[i] = x;
}

static ps_item heap_pop(ps_item *h, int64_t *n)
{
    const ps_item top = h[0];
    const ps_item x = h[--(*n)];
    int64_t i = 0;
    for (;;) {
        int64_t c = 2 * i + 1;
        if (c >= *n) break;
        if (c + 1 < *n && (h[c + 1].d < h[c].d || (h[c + 1].d == h[c].d && h[c + 1].v < h[c].v))) ++c;
        if (x.d < h[c].d || (x.d == h[c].d && x.v <= h[c].v)) break;
        h[i] = h[c];
        i = c;
    }
    if (*n > 0) h[i] = x;
    return top;
}

typedef struct {
    int64_t V, n_ports;
    const int32_t *port_off, *port_peer;
    const uint32_t *weight;
    const uint8_t *region;
} ps_graph;

/* weight of port p as a link, or 0 when it is none */
static int64_t ps_link(const ps_graph *g, int64_t p)
{
    const int64_t v = g->port_peer[p];
    if (v < 0 || v >= g->V) return 0;
    return g->weight ? (int64_t)g->weight[p] : 1;
}

/* one leg s -> t: number of links (path in buf[0..hops], s first), or -1 */
static int64_t ps_leg(const ps_graph *g, uint32_t A, const int32_t *fb, int64_t Kf, int64_t s, int64_t t,
                      int64_t *dist, ps_item *heap, int64_t *buf)
{
    const int64_t V = g->V;
    if (!usable(g->region, A, fb, Kf, s) || !usable(g->region, A, fb, Kf, t)) return -1;
    for (int64_t v = 0; v < V; ++v) dist[v] = -1;
    int64_t hn = 0;
    dist[s] = 0;
    heap_push(heap, &hn, (ps_item){0, s});
    while (hn > 0) {
        const ps_item it = heap_pop(heap, &hn);
        if (it.d != dist[it.v]) continue; /* stale entry */
        const int64_t b = g->port_off[it.v], e = g->port_off[it.v + 1];
        if (!range_ok(b, e, g->n_ports)) continue;
        for (int64_t p = b; p < e; ++p) {
            const int64_t w = ps_link(g, p);
            if (w <= 0) continue;
            const int64_t u = g->port_peer[p];
            if (!usable(g->region, A, fb, Kf, u)) continue;
            if (it.d + w >= PS_DIST_LIMIT) continue; /* beyond the distance range: unreachable */
            if (dist[u] < 0 || it.d + w < dist[u]) {
                dist[u] = it.d + w;
                heap_push(heap, &hn, (ps_item){dist[u], u});
            }
        }
    }
    if (dist[t] < 0) return -1;
    /* walk back from t: predecessor = lowest-numbered u with a link u -> cur, dist(u) + w = dist(cur) */
    int64_t n = 0, cur = t;
    buf[n++] = cur;
    while (cur != s) {
        int64_t pred = -1;
        for (int64_t u = 0; u < V && pred < 0; ++u) {
            if (dist[u] < 0) continue;
            const int64_t b = g->port_off[u], e = g->port_off[u + 1];
            if (!range_ok(b, e, g->n_ports)) continue;
            for (int64_t p = b; p < e; ++p) {
                const int64_t w = ps_link(g, p);
                if (w > 0 && g->port_peer[p] == cur && dist[u] + w == dist[cur]) { pred = u; break; }
            }
        }
        cur = pred;
        buf[n++] = cur;
    }
    for (int64_t i = 0; i < n / 2; ++i) {
        const int64_t x = buf[i];
        buf[i] = buf[n - 1 - i];
        buf[n - 1 - i] = x;
    }
    return n - 1;
}

/* the port of u of least (weight, index) that links u -> v */
static int64_t ps_port(const ps_graph *g, int64_t u, int64_t v)
{
    const int64_t b = g->port_off[u];
    int64_t best = -1, bw = 0;
    for (int64_t p = b; p < g->port_off[u + 1]; ++p) {
        const int64_t w = ps_link(g, p);
        if (w > 0 && g->port_peer[p] == v && (best < 0 || w < bw)) { best = p - b; bw = w; }
    }
    return best;
}

void orc_synthesize(int64_t V, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                    const uint32_t *weight, const uint8_t *region, int64_t Q, const int32_t *src,
                    const int32_t *target, const uint32_t *allowed, const int32_t *via, int64_t Kv,
                    const int32_t *forbid, int64_t Kf, const uint32_t *key, const int32_t *out_port,
                    int64_t prio, int64_t max_hops, const int64_t *qidx, int64_t nq, int32_t *hops,
                    int32_t *path, o_rule *rules, uint32_t *err, int nthreads)
{
    set_threads(nthreads);
    const ps_graph g = {V, n_ports, port_off, port_peer, weight, region};
    const int64_t slots = max_hops + 1;
    for (int64_t v = 0; v < V; ++v) {
        if (region[v] >= 32) *err |= F_JUR;
        if (!range_ok(port_off[v], port_off[v + 1], n_ports)) *err |= F_OFFSETS;
    }
    for (int64_t p = 0; p < n_ports; ++p) {
        if (port_peer[p] < -1 || port_peer[p] >= V) *err |= F_SWITCH;
        if (weight && weight[p] == 0) *err |= F_GRAPH;
    }
    for (int64_t q = 0; q < Q; ++q) {
        const int64_t t = target[q];
        if (src[q] < 0 || src[q] >= V || t < 0 || t >= V) { *err |= F_SWITCH; continue; }
        if (range_ok(port_off[t], port_off[t + 1], n_ports) &&
            (out_port[q] < 0 || out_port[q] >= port_off[t + 1] - port_off[t]))
            *err |= F_ACTION;
    }
    for (int64_t i = 0; i < Q * Kv; ++i)
        if (via[i] < -1 || via[i] >= V) { *err |= F_SWITCH; break; }
    for (int64_t i = 0; i < Q * Kf; ++i)
        if (forbid[i] < -1 || forbid[i] >= V) { *err |= F_SWITCH; break; }
#pragma omp parallel
    {
        const size_t nv = (size_t)(V > 0 ? V : 1);
        int64_t *dist = (int64_t *)malloc(sizeof(int64_t) * nv);
        int64_t *buf = (int64_t *)malloc(sizeof(int64_t) * (nv + 1));
        int64_t *walk = (int64_t *)malloc(sizeof(int64_t) * (size_t)(slots + 1));
        ps_item *heap = (ps_item *)malloc(sizeof(ps_item) * (size_t)(n_ports + 2));
#pragma omp for schedule(dynamic, 1)
        for (int64_t k = 0; k < nq; ++k) {
            const int64_t q = qidx[k];
            int32_t *pk = path + k * slots;
            o_rule *rk = rules + k * slots;
            for (int64_t i = 0; i < slots; ++i) pk[i] = -1;
            memset(rk, 0, sizeof(o_rule) * (size_t)slots);
            hops[k] = -1;
            const int64_t s = src[q], t = target[q];
            if (s < 0 || s >= V || t < 0 || t >= V) continue;
            if (!range_ok(port_off[t], port_off[t + 1], n_ports) || out_port[q] < 0 ||
                out_port[q] >= port_off[t + 1] - port_off[t])
                continue;
            const int32_t *w = via + q * Kv;
            const int32_t *fb = forbid + q * Kf;
            int64_t m = 0;
            while (m < Kv && w[m] != -1) ++m;
            int64_t total = 0, from = s, ok = 1;
            walk[0] = s;
            for (int64_t leg = 0; leg <= m && ok; ++leg) {
                const int64_t to = leg < m ? w[leg] : t;
                if (to < 0 || to >= V) { ok = 0; break; }
                const int64_t d = ps_leg(&g, allowed[q], fb, Kf, from, to, dist, heap, buf);
                if (d < 0 || total + d > max_hops) { ok = 0; break; }
                for (int64_t i = 1; i <= d; ++i) walk[total + i] = buf[i];
                total += d;
                from = to;
            }
            if (!ok) continue;
            hops[k] = (int32_t)total;
            for (int64_t i = 0; i <= total; ++i) {
                pk[i] = (int32_t)walk[i];
                o_rule *r = &rk[i];
                for (int j = 0; j < 4; ++j) {
                    r->value[j] = key[q * 4 + j];
                    r->mask[j] = j < 3 ? 0xFFFFFFFFu : 0xFFu;
                }
                r->priority = (uint16_t)prio;
                r->action = (uint16_t)(i < total ? ps_port(&g, walk[i], walk[i + 1]) : out_port[q]);
            }
        }
        free(dist);
        free(buf);
        free(walk);
        free(heap);
    }
}

/* ------------------------------------------------------------------ A6
 * Per-intent verdict: pass iff every check of the intent passes (paper,
 * validator check definition); an unenforceable intent fails closed.
 *   compute (kind bit 0): the selector row admits at least one node
 *       (NO_FEASIBLE_NODE = 1); a hybrid intent's two placed endpoints must
 *       both be admitted (ENDPOINT_INFEASIBLE = 2).
 *   network (kind bit 1): at least one flow (NO_FLOW = 3, the no-op
 *       policy); every trace stays inside the allowed jurisdictions
 *       (LEAK = 4), ends in EGRESS (UNDELIVERED = 5) at the expected switch
 *       and port when given (WRONG_EGRESS = 6); with path constraints, it
 *       visits none of the intent's forbidden switches (FORBIDDEN_SWITCH =
 *       8) and every required waypoint (WAYPOINT_MISSED = 9) -- the checks
 *       over realised paths in the validator check definition.
 * The reason is the smallest failing code; compute reasons come first.
 * Bit 7 is added when the intent's reachability query found no compliant
 * path.  A record that points outside its arrays, or kind not in {1,2,3},
 * gives MALFORMED = 7 and F_INTENT.
 */
void orc_report(int64_t I, const o_intent *intents, int64_t rows, const uint64_t *feasible, int64_t W,
                const uint32_t *popcnt, int64_t N, const o_trace *traces, int64_t T,
                const o_expect *expect, const int32_t *reach, int64_t Q, const uint32_t *visit,
                const o_path_expect *pexp, uint64_t *pass, uint8_t *reason, o_summary *summary, uint32_t *err)
{
    memset(summary, 0, sizeof(*summary));
    for (int64_t w = 0; w < (I + 63) / 64; ++w) pass[w] = 0;
    for (int64_t i = 0; i < I; ++i) {
        const o_intent *it = &intents[i];
        const o_expect *ex = &expect[i];
        const int kind = it->kind;
        int malformed = (kind < 1 || kind > 3);
        if (!malformed && (kind & 1)) {
            if (it->sel_row < 0 || it->sel_row >= rows) malformed = 1;
            if (kind == 3 && (it->src_node < 0 || it->src_node >= N || it->dst_node < 0 || it->dst_node >= N))
                malformed = 1;
        }
        if (!malformed && (kind & 2)) {
            if (it->trace_begin < 0 || it->trace_end < it->trace_begin || it->trace_end > T) malformed = 1;
            if (ex->reach_q < -1 || ex->reach_q >= Q) malformed = 1;
        }
        int r = 0, flag = 0;
        if (malformed) {
            set_flag(err, F_INTENT);
            r = 7;
        } else {
            if (kind & 1) {
                const uint64_t *row = feasible + (int64_t)it->sel_row * W;
                if (popcnt[it->sel_row] == 0) r = 1;
                else if (kind == 3) {
                    const int a = (row[it->src_node >> 6] >> (it->src_node & 63)) & 1;
                    const int b = (row[it->dst_node >> 6] >> (it->dst_node & 63)) & 1;
                    if (!(a && b)) r = 2;
                }
            }
            if (kind & 2) {
                if (r == 0) {
                    if (it->trace_end == it->trace_begin) r = 3;
                    for (int64_t t = it->trace_begin; t < it->trace_end; ++t) {
                        const o_trace *tr = &traces[t];
                        int code = 0;
                        if (tr->jmask & ~it->allowed) code = 4;
                        else if (tr->state != O_EGRESS) code = 5;
                        else if ((ex->dst_switch >= 0 && tr->last_switch != ex->dst_switch) ||
                                 (ex->dst_port >= 0 && tr->last_port != ex->dst_port)) code = 6;
                        else if (visit && (visit[t] & pexp[i].forbid)) code = 8;
                        else if (visit && (visit[t] & pexp[i].must) != pexp[i].must) code = 9;
                        if (code && (r == 0 || code < r)) r = code;
                    }
                }
                if (ex->reach_q >= 0 && reach[ex->reach_q] < 0) flag = 1;
            }
        }
        reason[i] = (uint8_t)(r | (flag ? 0x80 : 0));
        if (r == 0) pass[i >> 6] |= (uint64_t)1 << (i & 63);
        summary->counts[kind & 3][r] += 1;
        summary->no_path[kind & 3] += flag;
    }
}

// C-ABI entry points of libpc: argument validation, context, scratch arena,
// and dispatch to the kernel modules.  See include/pc.h for the contract.
#include <new>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pc_internal.h"

int pc_set_error(pc_ctx *ctx, int code, const char *fmt, ...)
{
    if (ctx) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(ctx->msg, sizeof(ctx->msg), fmt, ap);
        va_end(ap);
    }
    return code;
}

// Grow a context-owned device buffer to at least `bytes` (contents are not kept).
static int ensure_buffer(pc_ctx *ctx, char **buf, size_t *cap, size_t bytes)
{
    if (bytes <= *cap) return PC_OK;
    if (getenv("PC_FAIL_ALLOC")) return pc_set_error(ctx, PC_ENOMEM, "scratch allocation refused (PC_FAIL_ALLOC)");
    size_t want = bytes + bytes / 8 + (1 << 20);
    if (*buf) {
        PC_HIP(ctx, hipDeviceSynchronize());
        PC_HIP(ctx, hipFree(*buf));
        *buf = nullptr;
        *cap = 0;
    }
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, want);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return pc_set_error(ctx, PC_ENOMEM, "scratch allocation of %zu bytes failed: %s", want,
                            hipGetErrorString(e));
    }
    *buf = static_cast<char *>(p);
    *cap = want;
    return PC_OK;
}

int pc_ensure_arena(pc_ctx *ctx, size_t bytes) { return ensure_buffer(ctx, &ctx->arena, &ctx->arena_bytes, bytes); }

int pc_ensure_aux(pc_ctx *ctx, size_t bytes) { return ensure_buffer(ctx, &ctx->aux, &ctx->aux_bytes, bytes); }

int pc_ensure_delta(pc_ctx *ctx, size_t bytes) { return ensure_buffer(ctx, &ctx->delta, &ctx->delta_bytes, bytes); }

int pc_ensure_tc_meta(pc_ctx *ctx, size_t bytes)
{
    const int rc = ensure_buffer(ctx, &ctx->tc_meta, &ctx->tc_meta_bytes, bytes);
    if (rc != PC_OK) ctx->tc_S = -1;
    return rc;
}

int pc_ensure_tc_filt(pc_ctx *ctx, size_t bytes)
{
    const int rc = ensure_buffer(ctx, &ctx->tc_filt, &ctx->tc_filt_bytes, bytes);
    if (rc != PC_OK) ctx->tc_S = -1;
    return rc;
}

static hipEvent_t take_event(pc_ctx *ctx)
{
    if (!ctx->ev_free.empty()) {
        hipEvent_t e = ctx->ev_free.back();
        ctx->ev_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    return e;
}

KernelTimer::KernelTimer(pc_ctx *c, const char *n, hipStream_t s) : ctx(c), name(n), stream(s)
{
    if (!ctx->prof) return;
    a = take_event(ctx);
    b = take_event(ctx);
    if (a && b) (void)hipEventRecord(a, stream);
}

KernelTimer::~KernelTimer()
{
    if (!ctx->prof || !a || !b) return;
    (void)hipEventRecord(b, stream);
    ctx->pending.push_back({name, a, b});
}

// Resolve recorded event pairs into the per-kernel tallies.
static int drain_profile(pc_ctx *ctx)
{
    for (auto &p : ctx->pending) {
        PC_HIP(ctx, hipEventSynchronize(p.b));
        float ms = 0.f;
        PC_HIP(ctx, hipEventElapsedTime(&ms, p.a, p.b));
        bool found = false;
        for (auto &t : ctx->tally)
            if (t.name == p.name) {
                t.launches += 1;
                t.ms += ms;
                found = true;
                break;
            }
        if (!found) ctx->tally.push_back({p.name, 1, static_cast<double>(ms)});
        ctx->ev_free.push_back(p.a);
        ctx->ev_free.push_back(p.b);
    }
    ctx->pending.clear();
    return PC_OK;
}

extern "C" {

int pc_profile(pc_ctx *ctx, int enable)
{
    if (!ctx) return PC_EINVAL;
    int rc = drain_profile(ctx);
    if (rc) return rc;
    ctx->tally.clear();
    ctx->prof = enable != 0;
    return PC_OK;
}

int pc_profile_read(pc_ctx *ctx, int idx, const char **name, int64_t *launches, double *total_ms)
{
    if (!ctx || !name || !launches || !total_ms) return PC_EINVAL;
    int rc = drain_profile(ctx);
    if (rc) return rc;
    if (idx < 0 || idx >= static_cast<int>(ctx->tally.size())) return PC_EINVAL;
    *name = ctx->tally[idx].name.c_str();
    *launches = ctx->tally[idx].launches;
    *total_ms = ctx->tally[idx].ms;
    return PC_OK;
}

int pc_version(void) { return PC_VERSION; }

int pc_trace_keep_tables(pc_ctx *ctx, int enable)
{
    if (!ctx) return PC_EINVAL;
    ctx->tc_keep = enable != 0;
    if (!ctx->tc_keep) ctx->tc_S = -1;  // nothing kept survives switching reuse off
    return PC_OK;
}

const char *pc_last_error(const pc_ctx *ctx) { return ctx ? ctx->msg : "null context"; }

int pc_create(pc_ctx **out, int device)
{
    if (!out) return PC_EINVAL;
    *out = nullptr;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return PC_EDEVICE;
    }
    if (device < 0 || device >= n) return PC_EINVAL;
    pc_ctx *ctx = new (std::nothrow) pc_ctx();
    if (!ctx) return PC_ENOMEM;
    ctx->device = device;
    if (hipSetDevice(device) != hipSuccess ||
        hipMalloc(reinterpret_cast<void **>(&ctx->d_err), 256) != hipSuccess ||
        hipMemset(ctx->d_err, 0, 256) != hipSuccess ||
        hipMalloc(reinterpret_cast<void **>(&ctx->d_small), 256) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void **>(&ctx->h_small), 256, hipHostMallocDefault) != hipSuccess ||
        hipEventCreateWithFlags(&ctx->lvl_ev[0], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ctx->lvl_ev[1], hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        pc_destroy(ctx);
        return PC_EDEVICE;
    }
    if (pc_noalloc_setup(ctx) != PC_OK) {  // this device's address of the fixed scratch, once per device
        (void)hipGetLastError();
        pc_destroy(ctx);
        return PC_EDEVICE;
    }
    *out = ctx;
    return PC_OK;
}

int pc_destroy(pc_ctx *ctx)
{
    if (!ctx) return PC_OK;
    (void)hipSetDevice(ctx->device);
    (void)hipDeviceSynchronize();
    if (ctx->arena) (void)hipFree(ctx->arena);
    if (ctx->aux) (void)hipFree(ctx->aux);
    if (ctx->delta) (void)hipFree(ctx->delta);
    if (ctx->tc_meta) (void)hipFree(ctx->tc_meta);
    if (ctx->tc_filt) (void)hipFree(ctx->tc_filt);
    if (ctx->d_err) (void)hipFree(ctx->d_err);
    if (ctx->d_small) (void)hipFree(ctx->d_small);
    if (ctx->h_small) (void)hipHostFree(ctx->h_small);
    for (auto e : ctx->lvl_ev)
        if (e) (void)hipEventDestroy(e);
    for (auto &p : ctx->pending) {
        (void)hipEventDestroy(p.a);
        (void)hipEventDestroy(p.b);
    }
    for (auto e : ctx->ev_free) (void)hipEventDestroy(e);
    delete ctx;
    return PC_OK;
}

int pc_data_errors(pc_ctx *ctx, void *stream, uint32_t *flags, int clear)
{
    if (!ctx || !flags) return pc_set_error(ctx, PC_EINVAL, "pc_data_errors: null argument");
    hipStream_t s = static_cast<hipStream_t>(stream);
    PC_HIP(ctx, hipSetDevice(ctx->device));
    PC_HIP(ctx, hipMemcpyAsync(ctx->h_small, ctx->d_err, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    PC_HIP(ctx, hipStreamSynchronize(s));
    *flags = static_cast<uint32_t>(ctx->h_small[0]);
    if (clear) {
        PC_HIP(ctx, hipMemsetAsync(ctx->d_err, 0, sizeof(uint32_t), s));
        PC_HIP(ctx, hipStreamSynchronize(s));
    }
    return PC_OK;
}

#define PC_REQUIRE(cond, ...)                                       \
    do {                                                            \
        if (!(cond)) return pc_set_error(ctx, PC_EINVAL, __VA_ARGS__); \
    } while (0)

int pc_eval_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                      const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                      void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_preds >= 0, "pc_eval_selectors: negative size (N=%d I=%d n_preds=%lld)", N,
               I, (long long)n_preds);
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_eval_selectors: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_eval_selectors: L=0 with predicates");
    PC_REQUIRE(I == 0 || (pred_off && popcnt), "pc_eval_selectors: null pred_off/popcnt");
    PC_REQUIRE(n_preds == 0 || preds, "pc_eval_selectors: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_eval_selectors: null labels");
    PC_REQUIRE(I == 0 || N == 0 || feasible, "pc_eval_selectors: null feasible");
    if (I == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_selectors(ctx, labels, N, L, pred_off, preds, n_preds, I, feasible, popcnt,
                         static_cast<hipStream_t>(stream));
}

int pc_eval_selectors_noalloc(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                              const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                              void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_preds >= 0, "pc_eval_selectors_noalloc: negative size (N=%d I=%d n_preds=%lld)",
               N, I, (long long)n_preds);
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_eval_selectors_noalloc: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_eval_selectors_noalloc: L=0 with predicates");
    PC_REQUIRE(I == 0 || (pred_off && popcnt), "pc_eval_selectors_noalloc: null pred_off/popcnt");
    PC_REQUIRE(n_preds == 0 || preds, "pc_eval_selectors_noalloc: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_eval_selectors_noalloc: null labels");
    PC_REQUIRE(I == 0 || N == 0 || feasible, "pc_eval_selectors_noalloc: null feasible");
    if (I == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_selectors_noalloc(ctx, labels, N, L, pred_off, preds, n_preds, I, feasible, popcnt,
                                 static_cast<hipStream_t>(stream));
}

int pc_eval_affinity(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *row_off,
                     int32_t I, const int32_t *term_off, int32_t n_terms, const pc_pred *preds, int64_t n_preds,
                     uint64_t *feasible, uint32_t *popcnt, uint8_t *unknown, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_terms >= 0 && n_preds >= 0,
               "pc_eval_affinity: negative size (N=%d I=%d n_terms=%d n_preds=%lld)", N, I, n_terms,
               (long long)n_preds);
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_eval_affinity: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_eval_affinity: L=0 with predicates");
    PC_REQUIRE(I == 0 || (row_off && popcnt && unknown), "pc_eval_affinity: null row_off/popcnt/unknown");
    PC_REQUIRE(term_off, "pc_eval_affinity: null term_off");
    PC_REQUIRE(n_preds == 0 || preds, "pc_eval_affinity: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_eval_affinity: null labels");
    PC_REQUIRE(I == 0 || N == 0 || feasible, "pc_eval_affinity: null feasible");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_affinity(ctx, labels, N, L, row_off, I, term_off, n_terms, preds, n_preds, feasible, popcnt,
                        unknown, static_cast<hipStream_t>(stream));
}

int pc_score_preferred(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const uint64_t *feasible,
                       const int32_t *row_off, int32_t I, const int32_t *term_off, int32_t n_terms,
                       const uint32_t *weight, const pc_pred *preds, int64_t n_preds, int32_t *best_node,
                       uint32_t *best_score, uint32_t *n_best, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_terms >= 0 && n_preds >= 0,
               "pc_score_preferred: negative size (N=%d I=%d n_terms=%d n_preds=%lld)", N, I, n_terms,
               (long long)n_preds);
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_score_preferred: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_score_preferred: L=0 with expressions");
    PC_REQUIRE(I == 0 || (row_off && best_node && best_score && n_best),
               "pc_score_preferred: null row_off/best_node/best_score/n_best");
    PC_REQUIRE(term_off, "pc_score_preferred: null term_off");
    PC_REQUIRE(n_terms == 0 || weight, "pc_score_preferred: null weight");
    PC_REQUIRE(n_preds == 0 || preds, "pc_score_preferred: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_score_preferred: null labels");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_preferred(ctx, labels, N, L, feasible, row_off, I, term_off, n_terms, weight, preds, n_preds,
                         best_node, best_score, n_best, static_cast<hipStream_t>(stream));
}

int pc_eval_selectors_count(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                            const pc_pred *preds, int64_t n_preds, int32_t I, uint32_t *popcnt, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_preds >= 0, "pc_eval_selectors_count: negative size");
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_eval_selectors_count: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_eval_selectors_count: L=0 with predicates");
    PC_REQUIRE(I == 0 || (pred_off && popcnt), "pc_eval_selectors_count: null pred_off/popcnt");
    PC_REQUIRE(n_preds == 0 || preds, "pc_eval_selectors_count: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_eval_selectors_count: null labels");
    if (I == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_selectors(ctx, labels, N, L, pred_off, preds, n_preds, I, nullptr, popcnt,
                         static_cast<hipStream_t>(stream));
}

int pc_probe_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                       const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *probe_row,
                       const int32_t *probe_node, int32_t P, uint8_t *bit, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_preds >= 0 && P >= 0, "pc_probe_selectors: negative size");
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_probe_selectors: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_probe_selectors: L=0 with predicates");
    PC_REQUIRE(I == 0 || pred_off, "pc_probe_selectors: null pred_off");
    PC_REQUIRE(n_preds == 0 || preds, "pc_probe_selectors: null preds");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_probe_selectors: null labels");
    PC_REQUIRE(P == 0 || (probe_row && probe_node && bit), "pc_probe_selectors: null probe arrays");
    if (I == 0 && P == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_probes(ctx, labels, N, L, pred_off, preds, n_preds, I, probe_row, probe_node, P, bit,
                      static_cast<hipStream_t>(stream));
}

int pc_update_nodes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                    const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *nodes, int32_t M,
                    uint64_t *feasible, uint32_t *popcnt, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(N >= 0 && I >= 0 && n_preds >= 0 && M >= 0, "pc_update_nodes: negative size");
    PC_REQUIRE(M <= PC_UPDATE_MAX_NODES, "pc_update_nodes: M=%d above %d", M, PC_UPDATE_MAX_NODES);
    PC_REQUIRE(L >= 0 && L <= 65535, "pc_update_nodes: L=%d out of [0, 65535]", L);
    PC_REQUIRE(L > 0 || n_preds == 0, "pc_update_nodes: L=0 with predicates");
    PC_REQUIRE(I == 0 || (pred_off && popcnt), "pc_update_nodes: null pred_off/popcnt");
    PC_REQUIRE(n_preds == 0 || preds, "pc_update_nodes: null preds");
    PC_REQUIRE(M == 0 || nodes, "pc_update_nodes: null nodes");
    PC_REQUIRE(N == 0 || L == 0 || labels, "pc_update_nodes: null labels");
    PC_REQUIRE(I == 0 || N == 0 || feasible, "pc_update_nodes: null feasible");
    if (I == 0 && M == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_update_nodes(ctx, labels, N, L, pred_off, preds, n_preds, I, nodes, M, feasible, popcnt,
                            static_cast<hipStream_t>(stream));
}

int pc_synthesize_paths(pc_ctx *ctx, int32_t V, const int32_t *port_off, const int32_t *port_peer,
                        int64_t n_ports, const uint32_t *weight, const uint8_t *region, int32_t Q,
                        const int32_t *src, const int32_t *target, const uint32_t *allowed, const int32_t *via,
                        int32_t Kv, const int32_t *forbid, int32_t Kf, const pc_key *key, const int32_t *out_port,
                        int32_t prio, int32_t max_hops, int32_t *hops, int32_t *path, pc_rule *rules, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(V >= 0 && Q >= 0 && n_ports >= 0, "pc_synthesize_paths: negative size");
    PC_REQUIRE(V <= PC_SYNTH_MAX_V, "pc_synthesize_paths: V=%d above %d", V, PC_SYNTH_MAX_V);
    PC_REQUIRE(n_ports < (int64_t(1) << 31), "pc_synthesize_paths: n_ports too large");
    PC_REQUIRE(Kv >= 0 && Kv <= 32 && Kf >= 0 && Kf <= 32, "pc_synthesize_paths: Kv=%d / Kf=%d out of [0, 32]",
               Kv, Kf);
    PC_REQUIRE(max_hops >= 0 && max_hops <= 255, "pc_synthesize_paths: max_hops=%d out of [0, 255]", max_hops);
    PC_REQUIRE(prio >= 0 && prio <= 65535, "pc_synthesize_paths: prio=%d out of [0, 65535]", prio);
    PC_REQUIRE(V == 0 || (port_off && region), "pc_synthesize_paths: null port_off/region");
    PC_REQUIRE(n_ports == 0 || port_peer, "pc_synthesize_paths: null port_peer");
    PC_REQUIRE(Q == 0 || (src && target && allowed && key && out_port && hops && path && rules),
               "pc_synthesize_paths: null request or output array");
    PC_REQUIRE(Q == 0 || Kv == 0 || via, "pc_synthesize_paths: null via");
    PC_REQUIRE(Q == 0 || Kf == 0 || forbid, "pc_synthesize_paths: null forbid");
    if (Q == 0 && V == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_synthesize(ctx, V, port_off, port_peer, n_ports, weight, region, Q, src, target, allowed, via, Kv,
                          forbid, Kf, key, out_port, prio, max_hops, hops, path, rules,
                          static_cast<hipStream_t>(stream));
}

int pc_trace_flows(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                   const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
                   const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl, pc_trace_out *out,
                   void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(S >= 0 && T >= 0 && n_ports >= 0 && n_rules >= 0, "pc_trace_flows: negative size");
    PC_REQUIRE(ttl >= 0 && ttl <= 255, "pc_trace_flows: ttl=%d out of [0, 255]", ttl);
    PC_REQUIRE(n_rules < (int64_t(1) << 40), "pc_trace_flows: n_rules too large");
    PC_REQUIRE(T == 0 || (hdr && ingress && out), "pc_trace_flows: null hdr/ingress/out");
    PC_REQUIRE(S == 0 || (port_off && rule_off && jur), "pc_trace_flows: null topology array");
    PC_REQUIRE(n_ports == 0 || port_peer, "pc_trace_flows: null port_peer");
    PC_REQUIRE(n_rules == 0 || rules, "pc_trace_flows: null rules");
    if (T == 0 && S == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_trace(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, ingress, T, ttl,
                     nullptr, 0, out, nullptr, nullptr, nullptr, static_cast<hipStream_t>(stream));
}

int pc_trace_flows_watch(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer,
                         int64_t n_ports, const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules,
                         int64_t n_rules, const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl,
                         const int32_t *watch, int32_t K, pc_trace_out *out, uint32_t *visit, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(S >= 0 && T >= 0 && n_ports >= 0 && n_rules >= 0, "pc_trace_flows_watch: negative size");
    PC_REQUIRE(ttl >= 0 && ttl <= 255, "pc_trace_flows_watch: ttl=%d out of [0, 255]", ttl);
    PC_REQUIRE(K >= 0 && K <= 32, "pc_trace_flows_watch: K=%d out of [0, 32]", K);
    PC_REQUIRE(n_rules < (int64_t(1) << 40), "pc_trace_flows_watch: n_rules too large");
    PC_REQUIRE(T == 0 || (hdr && ingress && out && visit), "pc_trace_flows_watch: null hdr/ingress/out/visit");
    PC_REQUIRE(T == 0 || K == 0 || watch, "pc_trace_flows_watch: null watch");
    PC_REQUIRE(S == 0 || (port_off && rule_off && jur), "pc_trace_flows_watch: null topology array");
    PC_REQUIRE(n_ports == 0 || port_peer, "pc_trace_flows_watch: null port_peer");
    PC_REQUIRE(n_rules == 0 || rules, "pc_trace_flows_watch: null rules");
    if (T == 0 && S == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_trace(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, ingress, T, ttl,
                     watch, K, out, T ? visit : nullptr, nullptr, nullptr, static_cast<hipStream_t>(stream));
}

int pc_trace_flows_delta(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer,
                         int64_t n_ports, const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules,
                         int64_t n_rules, const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl,
                         const int32_t *changed, int32_t C, pc_trace_out *out, uint64_t *vsum, int32_t *walk,
                         int32_t *n_retraced, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(S >= 0 && T >= 0 && n_ports >= 0 && n_rules >= 0, "pc_trace_flows_delta: negative size");
    PC_REQUIRE(ttl >= 0 && ttl <= 255, "pc_trace_flows_delta: ttl=%d out of [0, 255]", ttl);
    PC_REQUIRE(n_rules < (int64_t(1) << 40), "pc_trace_flows_delta: n_rules too large");
    PC_REQUIRE(T == 0 || (hdr && ingress && out && vsum), "pc_trace_flows_delta: null hdr/ingress/out/vsum");
    PC_REQUIRE(n_retraced, "pc_trace_flows_delta: null n_retraced");
    PC_REQUIRE(C <= 0 || changed, "pc_trace_flows_delta: null changed");
    PC_REQUIRE(S == 0 || (port_off && rule_off && jur), "pc_trace_flows_delta: null topology array");
    PC_REQUIRE(n_ports == 0 || port_peer, "pc_trace_flows_delta: null port_peer");
    PC_REQUIRE(n_rules == 0 || rules, "pc_trace_flows_delta: null rules");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_trace_delta(ctx, S, port_off, port_peer, n_ports, jur, rule_off, rules, n_rules, hdr, ingress, T, ttl,
                           changed, C, out, vsum, walk, n_retraced, static_cast<hipStream_t>(stream));
}

int pc_masked_reach(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                    const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                    const int32_t *target, int32_t *dist, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(V >= 0 && Q >= 0 && n_adj >= 0, "pc_masked_reach: negative size");
    PC_REQUIRE(Q == 0 || (src && allowed && dist), "pc_masked_reach: null src/allowed/dist");
    PC_REQUIRE(V == 0 || (adj_off && region), "pc_masked_reach: null adj_off/region");
    PC_REQUIRE(n_adj == 0 || adj, "pc_masked_reach: null adj");
    if (Q == 0 && V == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_reach(ctx, V, adj_off, adj, n_adj, region, Q, src, allowed, target, dist,
                     static_cast<hipStream_t>(stream));
}

int pc_masked_reach_via(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                        const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                        const int32_t *target, const int32_t *via, int32_t Kv, const int32_t *forbid,
                        int32_t Kf, int32_t *dist, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(V >= 0 && Q >= 0 && n_adj >= 0, "pc_masked_reach_via: negative size");
    PC_REQUIRE(Kv >= 0 && Kv <= 32 && Kf >= 0 && Kf <= 32, "pc_masked_reach_via: Kv=%d Kf=%d out of [0, 32]", Kv,
               Kf);
    PC_REQUIRE(Q == 0 || (src && allowed && target && dist), "pc_masked_reach_via: null src/allowed/target/dist");
    PC_REQUIRE(Q == 0 || Kv == 0 || via, "pc_masked_reach_via: null via");
    PC_REQUIRE(Q == 0 || Kf == 0 || forbid, "pc_masked_reach_via: null forbid");
    PC_REQUIRE(V == 0 || (adj_off && region), "pc_masked_reach_via: null adj_off/region");
    PC_REQUIRE(n_adj == 0 || adj, "pc_masked_reach_via: null adj");
    if (Q == 0 && V == 0) return PC_OK;
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_reach_via(ctx, V, adj_off, adj, n_adj, region, Q, src, allowed, target, via, Kv, forbid, Kf, dist,
                         static_cast<hipStream_t>(stream));
}

int pc_report(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible,
              int32_t W, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
              const pc_flow_expect *expect, const int32_t *reach, int32_t Q, uint64_t *pass, uint8_t *reason,
              pc_summary *summary, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(I >= 0 && rows >= 0 && W >= 0 && N >= 0 && T >= 0 && Q >= 0, "pc_report: negative size");
    PC_REQUIRE(int64_t(W) * 64 >= N, "pc_report: W=%d too small for N=%d", W, N);
    PC_REQUIRE(summary, "pc_report: null summary");
    PC_REQUIRE(I == 0 || (intents && expect && pass && reason), "pc_report: null intent arrays");
    PC_REQUIRE(rows == 0 || (popcnt && (W == 0 || feasible)), "pc_report: null feasible/popcnt");
    PC_REQUIRE(T == 0 || traces, "pc_report: null traces");
    PC_REQUIRE(Q == 0 || reach, "pc_report: null reach");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_report(ctx, I, intents, rows, feasible, W, nullptr, popcnt, N, traces, T, expect, reach, Q, nullptr,
                      nullptr, pass, reason, summary, static_cast<hipStream_t>(stream));
}

int pc_report_counts(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint32_t *popcnt,
                     int32_t N, const uint8_t *ends, const pc_trace_out *traces, int32_t T,
                     const pc_flow_expect *expect, const int32_t *reach, int32_t Q, uint64_t *pass, uint8_t *reason,
                     pc_summary *summary, void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(I >= 0 && rows >= 0 && N >= 0 && T >= 0 && Q >= 0, "pc_report_counts: negative size");
    PC_REQUIRE(summary, "pc_report_counts: null summary");
    PC_REQUIRE(I == 0 || (intents && expect && pass && reason && ends), "pc_report_counts: null intent arrays");
    PC_REQUIRE(rows == 0 || popcnt, "pc_report_counts: null popcnt");
    PC_REQUIRE(T == 0 || traces, "pc_report_counts: null traces");
    PC_REQUIRE(Q == 0 || reach, "pc_report_counts: null reach");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_report(ctx, I, intents, rows, nullptr, 0, ends, popcnt, N, traces, T, expect, reach, Q, nullptr,
                      nullptr, pass, reason, summary, static_cast<hipStream_t>(stream));
}

int pc_report_paths(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible,
                    int32_t W, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
                    const pc_flow_expect *expect, const int32_t *reach, int32_t Q, const uint32_t *visit,
                    const pc_path_expect *pexp, uint64_t *pass, uint8_t *reason, pc_summary *summary,
                    void *stream)
{
    if (!ctx) return PC_EINVAL;
    ctx->msg[0] = 0;
    PC_REQUIRE(I >= 0 && rows >= 0 && W >= 0 && N >= 0 && T >= 0 && Q >= 0, "pc_report_paths: negative size");
    PC_REQUIRE(int64_t(W) * 64 >= N, "pc_report_paths: W=%d too small for N=%d", W, N);
    PC_REQUIRE(summary, "pc_report_paths: null summary");
    PC_REQUIRE(I == 0 || (intents && expect && pass && reason && pexp), "pc_report_paths: null intent arrays");
    PC_REQUIRE(rows == 0 || (popcnt && (W == 0 || feasible)), "pc_report_paths: null feasible/popcnt");
    PC_REQUIRE(T == 0 || (traces && visit), "pc_report_paths: null traces/visit");
    PC_REQUIRE(Q == 0 || reach, "pc_report_paths: null reach");
    PC_HIP(ctx, hipSetDevice(ctx->device));
    return run_report(ctx, I, intents, rows, feasible, W, nullptr, popcnt, N, traces, T, expect, reach, Q, visit, pexp,
                      pass, reason, summary, static_cast<hipStream_t>(stream));
}

}  // extern "C"

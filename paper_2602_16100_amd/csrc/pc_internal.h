// Internal declarations shared by the host layer and the kernel modules of
// libpc.  Not part of the public ABI (include/pc.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "pc.h"

struct pc_ctx {
    int device;
    char msg[512];
    uint32_t *d_err;     // sticky data-error word (device)
    int32_t *d_small;    // small device counters (live counts, totals)
    int32_t *h_small;    // pinned host mirror of d_small
    char *arena;         // scratch arena (device)
    size_t arena_bytes;
    char *aux;           // second scratch buffer, sized after a device-side count
    size_t aux_bytes;
    char *delta;         // compacted traces of an incremental re-trace (outside the arena it uses)
    size_t delta_bytes;
    // prepared tables kept between pc_trace_flows_delta calls: per-switch
    // group counts / offsets / prep-block offsets / action-error flags, and
    // the chunk sets; valid for tc_S switches and tc_groups groups
    char *tc_meta;
    size_t tc_meta_bytes;
    char *tc_filt;
    size_t tc_filt_bytes;
    int32_t tc_S = -1;
    int64_t tc_groups = 0;
    int64_t tc_blocks = 0;
    bool tc_keep = false;  // pc_trace_keep_tables: delta calls may reuse the kept tables
    hipEvent_t lvl_ev[2];  // trace level loop: completion of a level's live count copy
    // optional per-kernel timing (pc_profile)
    bool prof;
    std::vector<hipEvent_t> ev_free;
    struct Pending { const char *name; hipEvent_t a, b; };
    std::vector<Pending> pending;
    struct Tally { std::string name; int64_t launches; double ms; };
    std::vector<Tally> tally;
};

// Brackets the kernel launches in its scope with HIP events on `stream`
// when the context's profiling is enabled.
struct KernelTimer {
    pc_ctx *ctx;
    const char *name;
    hipStream_t stream;
    hipEvent_t a = nullptr, b = nullptr;
    KernelTimer(pc_ctx *c, const char *n, hipStream_t s);
    ~KernelTimer();
};

// Bump allocator over the context arena.  Sizes are computed first with a
// dry run (base == nullptr), then the arena is grown and carved for real.
struct Carver {
    char *base;
    size_t off;
    template <class T>
    T *take(size_t count, size_t align = 256)
    {
        off = (off + align - 1) / align * align;
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

int pc_set_error(pc_ctx *ctx, int code, const char *fmt, ...);
int pc_ensure_arena(pc_ctx *ctx, size_t bytes);
int pc_ensure_aux(pc_ctx *ctx, size_t bytes);
int pc_ensure_delta(pc_ctx *ctx, size_t bytes);
int pc_ensure_tc_meta(pc_ctx *ctx, size_t bytes);
int pc_ensure_tc_filt(pc_ctx *ctx, size_t bytes);

#define PC_HIP(ctx, expr)                                                                      \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return pc_set_error((ctx), PC_EDEVICE, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), \
                                __FILE__, __LINE__);                                           \
    } while (0)

#define PC_LAUNCH_CHECK(ctx) PC_HIP((ctx), hipGetLastError())

// Run a launch statement under a KernelTimer named after the kernel.
#define PC_TIMED(ctx, name, stream, ...)             \
    do {                                             \
        KernelTimer kt_((ctx), (name), (stream));    \
        __VA_ARGS__;                                 \
    } while (0)

// ---------------------------------------------------------------- common
void launch_fill_u32(uint32_t *p, size_t n, uint32_t v, hipStream_t s);
void launch_fill_u64(uint64_t *p, size_t n, uint64_t v, hipStream_t s);

// Exclusive scan of n int32 counts into out[0..n] (out[n] = total), one
// workgroup; optionally copies the result to out2 and clears counts.
void launch_scan_i32(const int32_t *counts, int32_t n, int32_t *out, int32_t *out2, int32_t *clear,
                     hipStream_t s);

// ---------------------------------------------------------------- modules
// fixed != nullptr: carve the scratch from fixed[0 .. fixed_cap) instead of
// the context's arena (PC_EINVAL, before any device work, if it does not fit)
int run_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                  const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                  hipStream_t stream, char *fixed = nullptr, size_t fixed_cap = 0);

// The allocation-free selector entry point's fixed scratch: pc_noalloc_setup
// (from pc_create, with ctx->device current) looks up this device's address
// of the array once; run_selectors_noalloc runs pc_eval_selectors on it.
int pc_noalloc_setup(pc_ctx *ctx);
int run_selectors_noalloc(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                          const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                          hipStream_t stream);

int run_affinity(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *row_off, int32_t I,
                 const int32_t *term_off, int32_t n_terms, const pc_pred *preds, int64_t n_preds, uint64_t *feasible,
                 uint32_t *popcnt, uint8_t *unknown, hipStream_t stream);
int run_preferred(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const uint64_t *feasible,
                  const int32_t *row_off, int32_t I, const int32_t *term_off, int32_t n_terms, const uint32_t *weight,
                  const pc_pred *preds, int64_t n_preds, int32_t *best, uint32_t *score, uint32_t *count,
                  hipStream_t stream);

// Flow tables already prepared for the trace engine: chunk sets and their
// per-switch group counts and offsets.
struct TracePrep {
    const uint32_t *filt;
    const int32_t *gcount;
    const int32_t *gofs;
    const uint32_t *cpos;  // per switch: the key nibbles its chunk sets filter on (5 bits each)
};

int run_trace(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
              const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
              const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl, const int32_t *watch, int32_t K,
              pc_trace_out *out, uint32_t *visit, uint64_t *vsum, int32_t *walk, hipStream_t stream,
              const TracePrep *pre = nullptr);

int run_trace_delta(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                    const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules, int64_t n_rules,
                    const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl, const int32_t *changed,
                    int32_t C, pc_trace_out *out, uint64_t *vsum, int32_t *walk, int32_t *n_retraced,
                    hipStream_t stream);

int run_reach(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
              const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
              const int32_t *target, int32_t *dist, hipStream_t stream);

int run_reach_via(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                  const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                  const int32_t *target, const int32_t *via, int32_t Kv, const int32_t *forbid, int32_t Kf,
                  int32_t *dist, hipStream_t stream);

int run_probes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
               const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *probe_row,
               const int32_t *probe_node, int32_t P, uint8_t *bit, hipStream_t stream);

int run_update_nodes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                     const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *nodes, int32_t M,
                     uint64_t *feasible, uint32_t *popcnt, hipStream_t stream);

int run_synthesize(pc_ctx *ctx, int32_t V, const int32_t *port_off, const int32_t *port_peer, int64_t n_ports,
                   const uint32_t *weight, const uint8_t *region, int32_t Q, const int32_t *src, const int32_t *target,
                   const uint32_t *allowed, const int32_t *via, int32_t Kv, const int32_t *forbid, int32_t Kf,
                   const pc_key *key, const int32_t *out_port, int32_t prio, int32_t max_hops, int32_t *hops,
                   int32_t *path, pc_rule *rules, hipStream_t stream);

int run_report(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible,
               int32_t W, const uint8_t *ends, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
               const pc_flow_expect *expect, const int32_t *reach, int32_t Q, const uint32_t *visit,
               const pc_path_expect *pexp, uint64_t *pass, uint8_t *reason, pc_summary *summary, hipStream_t stream);

// ---------------------------------------------------------------- device helpers
__device__ __forceinline__ bool pc_range_ok(int64_t b, int64_t e, int64_t n)
{
    return b >= 0 && e >= b && e <= n;
}

__device__ __forceinline__ int pc_lane() { return threadIdx.x & 63; }

__device__ __forceinline__ uint32_t pc_wave_sum_u32(uint32_t v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Map a linear block id onto work items so that each of the 8 XCDs (blocks
// are dealt to XCDs round-robin) receives one contiguous range of items.
__device__ __forceinline__ int64_t pc_xcd_item(int64_t total)
{
    const int64_t per = (total + 7) / 8;
    const int64_t b = blockIdx.x;
    return (b & 7) * per + (b >> 3);
}

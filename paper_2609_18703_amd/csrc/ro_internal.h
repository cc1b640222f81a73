// Internal declarations shared by the host runtime and the kernel sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ro.h"

namespace ro {

constexpr int kBlock = 256;                 // threads per workgroup (4 waves of 64)
constexpr int kItems = 16;                  // items per thread in scan tiles
constexpr int kTile = kBlock * kItems;      // 4096 entries per scan tile
constexpr int kSub = 256;                   // children per copy sub-tile (the scan records where each starts)
constexpr int kCntLds = 512;                // parents whose counts a tile aggregates in LDS

// Canonical per-child record written by the report scatter.  `tag` holds the
// call epoch (bits 31..2) and the terminal state (bits 1..0): an entry is
// valid for the current call only if its epoch matches, so the array never
// needs clearing between calls.
struct alignas(16) Canon {
    uint64_t src;     // device address of the record's first byte
    uint32_t len;     // bytes copied (0 unless SUCCESS)
    uint32_t tag;     // epoch << 2 | state
};
static_assert(sizeof(Canon) == 16, "Canon must be 16 bytes");

// Device-resident control words of one context.
struct Ctl {
    int32_t err;             // first error (0 = none)
    uint32_t done;           // workgroups finished (ticketed kernels)
    uint64_t ticket;         // next tile ticket (ticketed kernels)
    int64_t n_valid;         // gather: accepted (non-pending) reports of this call
    int64_t n_filled;        // gather: canonical slots holding this call's epoch
    int64_t total;           // gather / emit: total bytes
    int64_t n_items;         // emit: emitted parents
    int64_t n_virtual;       // emit: children of emitted parents
    int64_t n_rejected;      // gather: reports rejected by a group-failure barrier
    uint32_t scan_epoch;     // look-back descriptor epoch of the next ticketed launch (1..65535)
    uint32_t pad32;
    int64_t pad[7];
};

struct Tracer;

struct Launch {
    hipStream_t stream;
    int num_cus;
    Ctl *ctl;
    uint64_t *desc;          // look-back descriptors
    int64_t desc_cap;        // tiles
    Tracer *tracer;          // per-kernel events, or null
};

// Bracket one kernel launch with trace events when tracing is on.
void trace_begin(const Launch &L, int kernel);
void trace_end(const Launch &L, int kernel);

#define RO_LAUNCH(L, kid, ...)               \
    do {                                     \
        ::ro::trace_begin((L), (kid));       \
        hipLaunchKernelGGL(__VA_ARGS__);     \
        ::ro::trace_end((L), (kid));         \
    } while (0)

constexpr uint32_t kMaxScanEpoch = 65535;
constexpr uint32_t kMaxCanonEpoch = (1u << 30) - 1;

hipError_t launch_clear_err(const Launch &L);
hipError_t launch_ctl_init(const Launch &L);
hipError_t launch_zero_u64(const Launch &L, uint64_t *p, int64_t n);
hipError_t launch_clear_tags(const Launch &L, Canon *canon, int64_t n);

// ---- launchers (defined in the kernel sources) ----------------------------
hipError_t launch_expand(const Launch &L, const int32_t *counts, int64_t P,
                         int64_t *offsets, uint32_t *child_parent, uint32_t *child_ordinal,
                         int64_t child_cap);

// cpar (or null): the parent of each of the first cpar_n children, which
// then replaces the search of the offsets (a stream's own map); ids past
// cpar_n are out of range
hipError_t launch_batch(const Launch &L, const uint32_t *queue, const uint8_t *keep,
                        int64_t Q, const int64_t *offsets, int64_t P, int32_t B,
                        uint32_t *out_child, uint32_t *out_parent, uint32_t *out_ordinal,
                        int64_t out_cap, int64_t *n_out, int64_t *n_batches, uint32_t *cmap,
                        int64_t cmap_cap, const uint8_t *barrier, const uint32_t *cpar = nullptr,
                        int64_t cpar_n = 0);
hipError_t launch_expand_tags(const Launch &L, const int64_t *offsets, int64_t P, uint32_t *child_parent,
                              uint32_t *child_ordinal, int64_t child_cap);

// parent-bound reservation workspace ([cap] queue entries, [pcap] parents)
struct PbWs {
    uint32_t *kc;            // ready children in queue order
    uint32_t *k[2];          // sort keys (parents), double-buffered
    uint64_t *v[2];          // sort values (child << 32 | queue position), double-buffered
    uint32_t *fsize;         // per queue position: group size if a group's first entry, else 0
    uint32_t *bidx;          // per group-first position: batch number
    uint32_t *pstart, *pend; // per parent: sorted index range
    int32_t *hist;           // digit histograms, [buckets * tiles]
    int64_t *hoff;           // their exclusive scan
    int64_t *m;              // [2] ready count, scratch
};
hipError_t launch_batch_parent(const Launch &L, const uint32_t *queue, const uint8_t *keep, int64_t Q,
                               const int64_t *offsets, int64_t P, int32_t B, uint32_t *out_child,
                               uint32_t *out_parent, uint32_t *out_ordinal, int64_t out_cap, int64_t *batch_off,
                               int64_t batch_cap, int64_t *n_out, int64_t *n_batches, uint32_t *cmap,
                               int64_t cmap_cap, const uint8_t *barrier, const PbWs &w);
constexpr int64_t kPbTile = 2048;        // sort tile
constexpr int64_t kPbSpan = 8;           // sort tiles per histogram column
constexpr int64_t kPbMaxBuckets = 512;

struct GatherArgs {
    const uint32_t *rp, *ro;
    const uint8_t *rs;
    const int64_t *roff;
    const uint8_t *data;
    int64_t n;
    const int64_t *offsets;
    int64_t P;
    int64_t *out_off;
    uint8_t *out_data;
    int64_t out_cap;
    int32_t *ns, *nf, *nk;
    uint8_t *complete, *pstate;
    int64_t *cdst;           // per-child output positions (or null)
    uint8_t *barrier;        // group-failure barrier of the Call (or null)
    int64_t *n_rejected;     // device scalar (or null)
};

struct GatherWs {
    Canon *canon;
    int64_t canon_cap;
    int64_t *sub_base;       // per copy sub-tile: first output byte
    int64_t sub_cap;
    uint64_t *gkey;          // [P] first group failure per parent (epoch << 32 | ~report index)
};

// epoch: the canonical epoch of this gather (kept by the host: 1..2^30-1,
// one more per gather, every slot tag cleared when it wraps), which tags its
// slots and its group-failure keys
hipError_t launch_gather(const Launch &L, const GatherArgs &a, const GatherWs &w, uint32_t epoch);

// grain phases and the generation fence.  One 16-byte record per Grain:
// word = phase (READY or IN-FLIGHT) | generation << 32, changed by one 64-bit
// compare-and-swap; key = the accepted report, epoch << 32 | ~index, of the
// commit call that sealed the Grain (0 while unsealed).  A report touches one
// record: one random access.
struct alignas(16) Grain {
    uint64_t word;
    uint64_t key;
};
static_assert(sizeof(Grain) == 16, "grain record");
hipError_t launch_grains_fill(const Launch &L, Grain *g, int64_t n);
hipError_t launch_grains_rekey(const Launch &L, Grain *g, int64_t n);
hipError_t launch_grains_read(const Launch &L, const Grain *g, int64_t n, uint32_t *phase, uint32_t *gen);
hipError_t launch_grains_dispatch(const Launch &L, const uint32_t *child, int64_t n, int64_t N, Grain *g,
                                  uint32_t *out_gen);
hipError_t launch_grains_retry(const Launch &L, const uint32_t *child, int64_t n, int64_t N, Grain *g);
hipError_t launch_grains_commit(const Launch &L, const uint32_t *rp, const uint32_t *ro, const uint8_t *rs,
                                const int64_t *roff, const uint8_t *data, const uint32_t *rgen, int64_t n,
                                const int64_t *offsets, int64_t P, int64_t N, Grain *g, uint32_t epoch, uint32_t *tag,
                                uint8_t *state_out, int64_t *counts);
hipError_t launch_grains_zero_tags(const Launch &L, uint32_t *tag, int64_t n);

// filter / broadcast
constexpr int kMaxBroadcastLevels = 8;
hipError_t launch_filter(const Launch &L, const uint8_t *xs, const uint8_t *ms, const uint8_t *mv, int64_t n,
                         uint8_t *out);
hipError_t launch_broadcast(const Launch &L, const uint32_t *const *maps, const int64_t *map_len, int32_t levels,
                            int64_t n, const uint8_t *xs, int64_t n_anc, const uint8_t *ls, uint32_t *anc,
                            uint8_t *out);

// streaming
struct StreamState {
    const int64_t *offsets;
    int64_t P, N;
    Canon *canon;            // [N] accepted reports (tag epoch 1 = accepted)
    uint32_t *seen;          // [N/32] duplicate detection bitmap
    int32_t *mid;            // [stream_mid_size(N)] report counters of parents with 64..1023 children
    int32_t *big;            // [stream_big_size(N)] spread report counters of large parents
    uint8_t *emitted;        // [P]
    int64_t *ebase;          // [P] per emitted parent: canonical slot of its first child minus evoff
    int64_t *evoff;          // [P+1] child offsets of the emitted parents (virtual children)
    int32_t *ecnt;           // [3*(P+1)] SUCCESS / FAILED / SKIPPED counts per emitted parent
    int64_t *edst;           // [N+1] output position of each virtual child
    uint64_t *esrc;          // [N] source address of each virtual child's bytes
    uint8_t *barrier;        // [P] the Call's group-failure barrier (caller's, or null)
    uint64_t *gkey;          // [P] first group failure per parent in the current report call
    uint8_t *ebar;           // [P] per emitted parent: barred
    uint32_t *cpar;          // [N] parent of every child (for the stream's batches)
    uint32_t run_epoch;      // slot tag epoch of this run (advanced by each reset)
    uint32_t gf_epoch;       // epoch of the current report call in gkey
};

// First group-failure report of each parent among reports [0, n), as the
// largest key (epoch << 32 | ~i); reports of parents already barred are
// skipped.  Then, after the commit pass, set the barrier of every parent
// whose first group failure is in this call.
hipError_t launch_first_gf(const Launch &L, const uint8_t *rs, const uint32_t *rp, int64_t n, int64_t P,
                           const uint8_t *barrier, uint64_t *gkey, uint32_t epoch);
hipError_t launch_gf_fold(const Launch &L, const uint8_t *rs, const uint32_t *rp, int64_t n, int64_t P,
                          uint8_t *barrier, const uint64_t *gkey, uint32_t epoch);

int64_t stream_mid_size(int64_t N);
int64_t stream_big_size(int64_t N);
int64_t stream_desc_tiles(int64_t P, int64_t N);
hipError_t launch_stream_init(const Launch &L, StreamState &s);
hipError_t launch_stream_reset(const Launch &L, StreamState &s);
hipError_t launch_stream_report(const Launch &L, StreamState &s, const uint32_t *rp,
                                const uint32_t *ro, const uint8_t *rs, const int64_t *roff,
                                const uint8_t *data, int64_t n, int64_t *n_rejected);
hipError_t launch_stream_emit(const Launch &L, StreamState &s,
                              uint32_t *emit_parent, int64_t *emit_off, uint8_t *emit_data,
                              int64_t cap_parents, int64_t cap_bytes, int32_t *ns, int32_t *nf,
                              int32_t *nk, uint8_t *pstate, int64_t *n_emitted, int64_t *n_bytes);

}  // namespace ro

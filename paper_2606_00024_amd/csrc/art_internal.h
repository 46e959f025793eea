// Internal declarations shared by the host API (art_api.cpp) and the kernels
// (art_kernels.hip).  Not part of the public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace art {

constexpr int kHeadDim = 128;   // dims per head (the only supported value)
constexpr int kTile = 64;       // tokens one wavefront processes per tile
constexpr int kWaves = 4;       // wavefronts per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxChunkTiles = 16;   // tiles one loader streams per chunk (and per block)
constexpr int kMaxChunkBlocks = 16;  // blocks per chunk
// Work-list indices live in the low 24 bits of the queue word; a launch
// hands out at most its list length plus one final index per workgroup.
constexpr int kQueueBits = 24;
constexpr int64_t kQueueSlack = 1 << 16;
// The work list is split over this many queue words (each run of kQueues
// groups spread over all of them), each in its own 256-byte line.
constexpr int kQueues = 8;
constexpr int kQueueStride = 32;  // uint64 words between queue words

// Progress of one chunk, published in bits 20..22 of its flag word (the
// call's epoch is in bits 24..63, bits 0..19 carry the stability summary or
// state).  States only ever increase.
enum ChunkState : uint32_t {
    kNone = 0,
    kAggregate = 1,      // softmax aggregate of the chunk's own blocks
    kInclusive = 2,      // softmax state after the chunk (inclusive prefix)
    kStabSummary = 3,    // stability summary of the chunk's own blocks
    kStabInclusive = 4,  // stop/patience state after the chunk
};

// Byte layout of a workspace (all offsets from its start, 256-aligned).
struct WorkspaceLayout {
    size_t error_off;        // uint64 error word: 0, or epoch << 8 | status of the call that gave up
    size_t queue_off;        // kQueues work-queue words (one per 256 bytes): epoch << 24 | next index
    size_t stop_off;         // uint64 [groups] announced stop: epoch << 24 | chunk
    size_t flags_off;        // uint64 [groups][max_chunks]: epoch << 24 | state << 20 | payload
    size_t records_off;      // float [groups][max_chunks][2][record_floats]
    size_t head_off;         // per-head mode: int32 [groups][max_chunks][g][8]; else 0 bytes
    size_t total;
};

struct Plan {
    int32_t group;           // query heads per KV head (g)
    int32_t tiles_per_block; // block_size / kTile
    int32_t chunk_blocks;    // blocks per chunk (C)
    int32_t lead_chunks;     // leading chunks of a traversal that hold lead_blocks blocks
    int32_t lead_blocks;
    int32_t max_chunks;      // chunks per group the grid provides
    int32_t n_groups;        // batch * num_kv_heads
    int32_t t_cap;           // traversal length bound per group
    int32_t record_floats;   // floats per aggregate / inclusive record
    int32_t loader_partials; // see KernelParams
    int32_t v_in_record;     // see KernelParams
    int32_t slots;           // chunk buffers in LDS (2 or 3)
    size_t lds_bytes;        // dynamic LDS per workgroup
    WorkspaceLayout ws;
};

// Everything the kernel reads, passed by value.
struct KernelParams {
    // shape
    int32_t batch, num_q_heads, num_kv_heads, block_size, page_shift, num_pages;
    int32_t max_pages, max_list, list_per_head;
    int64_t ks_page, ks_head, ks_tok, vs_page, vs_head, vs_tok;
    // options
    float scale_log2;        // softmax_scale * log2(e): scores kept in base 2
    float tau, phi;
    int32_t patience, dense_order, out_bf16;
    int32_t probe_stride;    // the stability test sees coordinates 0, s, 2s, ... (1 = all)
    int32_t scale_of_accumulator;  // 1: d_scale on the unnormalised accumulator L o
    int32_t no_detector;     // 1: no stability test at all (full attention over the traversal)
    int32_t per_head;        // 1: every query head has its own patience counter and stop
    // plan
    int32_t tiles_per_block, chunk_blocks, max_chunks, t_cap, record_floats;
    int32_t lead_chunks, lead_blocks;  // the first lead_chunks chunks hold lead_blocks blocks
    int32_t work_chunks;     // chunk rows of the work list (<= max_chunks)
    int32_t chunk_recs_lds;  // block records per LDS chunk buffer
    int32_t loader_partials; // per-loader partial aggregates kept in LDS (3 or 0)
    int32_t n_slots;         // chunk buffers in LDS (2 or 3)
    int32_t v_in_record;     // 1: V is staged in the LDS record being written (no staging buffers)
    int32_t look_first;      // 1: a chunk looks back once before publishing its aggregate (set at launch)
    // data
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* page_table;
    const int32_t* seq_lens;
    const int32_t* block_list;
    const int32_t* block_list_len;
    void* out;
    float* lse;
    int32_t* stop_block;
    // workspace
    uint64_t* error_word;
    uint64_t* queue;
    uint64_t* stop_word;
    uint64_t* flags;
    float* records;
    int32_t* head_area;      // per-head mode: [groups][max_chunks][g][8] int32
    uint64_t epoch;          // unique per call; tags every flag it writes
    uint32_t spin_limit;     // polls before a wait gives up
    int32_t max_ahead;       // 0, or chunks a load may run ahead of the last tested chunk
};

// Launchers (art_kernels.hip).  Return a hipError_t.
int launch_decode(const Plan& plan, const KernelParams& params, hipStream_t stream);
int launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);
// Device address of the library's static scratch on the current device
// (art_static.hip); set up (address taken, zero-filled on `stream`) on the
// first call per device.  Returns a hipError_t.
int static_scratch(hipStream_t stream, void** ptr);

}  // namespace art

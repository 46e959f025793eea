// Host side of the C ABI declared in include/art.h: argument checks, the
// launch plan (a function of the shape only), the workspace layout, the
// per-call epoch and the checked-mode validator.
#include "art.h"

#include <math.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <random>
#include <vector>

#include "art_internal.h"

namespace {

using art::Plan;
using art::KernelParams;

constexpr size_t kAlign = 256;
constexpr uint32_t kSpinLimit = 1u << 22;  // polls (~seconds) before a wait gives up

// Process-wide call counter: every launch tags the flags it writes with a
// fresh value, so flags left by earlier calls are never mistaken for current.
// It starts at a random point of [2^38, 2^39): the words of a workspace that
// earlier held another layout (small integers, float bits) cannot pass for a
// current tag, and 2^39 calls remain before the 2^40 limit of the tags.
uint64_t initial_epoch() {
    std::random_device rd;
    uint64_t r = ((uint64_t)rd() << 32) ^ rd();
    r ^= (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    return (uint64_t(1) << 38) | (r & ((uint64_t(1) << 38) - 1));
}

uint64_t next_epoch() {
    static std::atomic<uint64_t> counter{initial_epoch()};
    return counter.fetch_add(1, std::memory_order_relaxed);
}

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

constexpr int kLeadChunks = 4;  // leading short chunks per traversal
constexpr int kLeadBlocks = 3;  // blocks in each of them

// Chunks of a traversal of T blocks (the kernel's chunks_for).
int64_t chunks_for(int64_t T, int C, int lead_chunks, int lead_blocks) {
    const int64_t lead_T = (int64_t)lead_chunks * lead_blocks;
    return T <= lead_T ? (T + lead_blocks - 1) / lead_blocks : lead_chunks + (T - lead_T + C - 1) / C;
}

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

int ilog2(int64_t x) {
    int r = 0;
    while ((int64_t(1) << r) < x) ++r;
    return r;
}

art_status check_shape(const art_decode_shape* s, const art_decode_opts* o) {
    if (!s || !o) return ART_ERR_INVALID_ARG;
    if (s->batch < 0 || s->num_kv_heads <= 0 || s->num_q_heads <= 0 ||
        s->num_q_heads % s->num_kv_heads != 0 || s->head_dim <= 0 || s->block_size <= 0 ||
        s->page_size <= 0 || s->num_pages <= 0 || s->max_pages_per_seq <= 0 ||
        s->max_blocks_per_list < 0 || (s->list_per_head != 0 && s->list_per_head != 1))
        return ART_ERR_INVALID_ARG;
    if (s->k_stride_page < 0 || s->k_stride_head < 0 || s->k_stride_token < 0 ||
        s->v_stride_page < 0 || s->v_stride_head < 0 || s->v_stride_token < 0)
        return ART_ERR_INVALID_ARG;
    if (isnan(o->tau) || isnan(o->phi) || !isfinite(o->softmax_scale) || o->patience < 1 ||
        (o->dense_order != ART_ORDER_RECENT_FIRST && o->dense_order != ART_ORDER_FORWARD) ||
        (o->out_dtype != ART_OUT_F32 && o->out_dtype != ART_OUT_BF16) || o->chunk_blocks < 0 ||
        o->chunk_blocks > art::kMaxChunkBlocks || o->probe_stride < 0 ||
        (o->probe_stride & (o->probe_stride - 1)) != 0 ||
        (o->probe_stride > 1 && s->head_dim % o->probe_stride != 0) ||
        (o->scale_of_accumulator != 0 && o->scale_of_accumulator != 1) ||
        (o->no_detector != 0 && o->no_detector != 1) || o->max_wait_polls < 0 ||
        (o->per_head_stop != 0 && o->per_head_stop != 1) || o->max_ahead_chunks < 0)
        return ART_ERR_INVALID_ARG;
    const int g = s->num_q_heads / s->num_kv_heads;
    if (s->head_dim != art::kHeadDim) return ART_ERR_UNSUPPORTED;
    if (g != 1 && g != 2 && g != 4 && g != 8 && g != 16) return ART_ERR_UNSUPPORTED;
    if (s->block_size % art::kTile != 0 || s->block_size / art::kTile > art::kMaxChunkTiles)
        return ART_ERR_UNSUPPORTED;
    if (!is_pow2(s->page_size) || s->page_size < 16) return ART_ERR_UNSUPPORTED;
    // 16-byte vector loads of 8 head dims need 8-element aligned rows
    if (s->k_stride_page % 8 || s->k_stride_head % 8 || s->k_stride_token % 8 ||
        s->v_stride_page % 8 || s->v_stride_head % 8 || s->v_stride_token % 8)
        return ART_ERR_UNSUPPORTED;
    return ART_OK;
}

// Everything about the launch is decided here from the shape (and the
// chunk_blocks option): never from the data or the thresholds.
art_status make_plan(const art_decode_shape* s, const art_decode_opts* o, Plan* p) {
    art_status st = check_shape(s, o);
    if (st != ART_OK) return st;
    const int g = s->num_q_heads / s->num_kv_heads;
    const int tpb = s->block_size / art::kTile;
    const int64_t cap_tokens = (int64_t)s->max_pages_per_seq * s->page_size;
    const int64_t t_dense = (cap_tokens + s->block_size - 1) / s->block_size;
    int64_t t_cap = t_dense > s->max_blocks_per_list ? t_dense : s->max_blocks_per_list;
    if (t_cap < 1) t_cap = 1;
    // stability runs travel in 19 bits of a flag word
    if (t_cap >= (int64_t(1) << 19)) return ART_ERR_UNSUPPORTED;
    const int64_t n_groups = (int64_t)s->batch * s->num_kv_heads;

    // LDS of a workgroup: two or three chunk buffers of C*tpb tile records
    // plus three per-loader partial aggregates each (when they fit), and
    // three V staging buffers: half tiles (32 rows of 288 bytes) for groups
    // of up to 4 heads, quarter tiles (4 KiB) for 8 or more.  A record of 8
    // or more heads holds 4 KiB of outputs, so when every block is one tile
    // the loaders stage V in the record the tile is about to write, and the
    // staging buffers go.
    // Kept within 78 KiB, so that two workgroups share a CU's 160 KiB.
    const size_t rec_bytes = (size_t)(g * art::kHeadDim + 2 * g) * 4;
    const bool v_in_record = g >= 8 && tpb == 1;
    const size_t pbuf_bytes = v_in_record ? 0 : (g >= 8 ? (size_t)3 * 4096 : (size_t)3 * 32 * 288) + 16;
    const size_t lds_cap = 78 * 1024;
    auto lds_for = [&](int blocks, int partials, int slots = 2) {
        return slots * (size_t)(blocks + partials) * rec_bytes + pbuf_bytes;
    };
    // the per-loader partials save the resolver a fold over the blocks; they
    // are kept unless dropping them lets a chunk hold more blocks (up to 8)
    auto blocks_fitting = [&](int partials) {
        int b = art::kMaxChunkBlocks;
        while (b > 0 && lds_for(b, partials) > lds_cap) --b;
        return b;
    };
    const int b3 = blocks_fitting(3), b0 = blocks_fitting(0);
    const int partials = (b3 >= 1 && b3 >= (b0 < 8 ? b0 : 8)) ? 3 : 0;
    int c_max = partials ? b3 : b0;
    // a loader streams at most kMaxChunkTiles tiles of a chunk
    while (c_max > 1 && (c_max + 2) / 3 * tpb > art::kMaxChunkTiles) --c_max;
    if (c_max < 1) return ART_ERR_UNSUPPORTED;

    int C;
    if (o->chunk_blocks > 0) {
        C = o->chunk_blocks;
    } else {
        // up to 9 blocks per chunk, a multiple of the three loaders when the
        // budget allows; 6, then 3, only when the whole problem has fewer
        // than 64 chunks.  (Measured: halving the chunk whenever there were
        // fewer chunks than 1024 cost 17-210 % on problems of 2 to 16
        // groups; the per-chunk work of the resolver outweighs the wider
        // spread.)
        C = c_max < 9 ? c_max : 9;
        if (C >= 3) C -= C % 3;
        while (C > 3 && n_groups * ((t_cap + C - 1) / C) < 64) C -= 3;
        // the work list must fit a queue word
        while (C < c_max && n_groups * ((t_cap + C - 1) / C) + art::kQueueSlack >= (1 << art::kQueueBits)) C *= 2;
    }
    if (C > c_max) C = c_max;
    if (C < 1) C = 1;
    // Leading chunks of kLeadBlocks blocks: the first decisions of every
    // group come sooner, so that groups that stop early claim less past
    // their stop (only with the default chunk size).
    int lead_chunks = 0, lead_blocks = C;
    if (o->chunk_blocks == 0 && C > kLeadBlocks) {
        lead_chunks = kLeadChunks;
        lead_blocks = kLeadBlocks;
    }
    p->lead_chunks = lead_chunks;
    p->lead_blocks = lead_blocks;
    const int64_t max_chunks = chunks_for(t_cap, C, lead_chunks, lead_blocks);
    if (n_groups * max_chunks + art::kQueueSlack >= (1 << art::kQueueBits)) return ART_ERR_UNSUPPORTED;

    p->group = g;
    p->tiles_per_block = tpb;
    p->chunk_blocks = C;
    p->max_chunks = (int32_t)max_chunks;
    p->n_groups = (int32_t)n_groups;
    p->t_cap = (int32_t)t_cap;
    p->record_floats = (g * art::kHeadDim + 2 * g + 63) / 64 * 64;
    p->loader_partials = partials;
    p->v_in_record = v_in_record ? 1 : 0;
    // (a third buffer was measured: it lets loaders run further past a
    // stop and gains nothing elsewhere)
    p->slots = 2;
    p->lds_bytes = lds_for(C, partials, p->slots);

    art::WorkspaceLayout& w = p->ws;
    size_t off = 0;
    w.error_off = off;      off = align_up(off + 8);
    w.queue_off = off;      off = align_up(off + 8 * art::kQueueStride * art::kQueues);
    w.stop_off = off;       off = align_up(off + 8 * (size_t)n_groups);
    w.flags_off = off;      off = align_up(off + 8 * (size_t)n_groups * max_chunks);
    w.records_off = off;    off = align_up(off + (size_t)n_groups * max_chunks * 2 * p->record_floats * 4);
    w.head_off = off;
    if (o->per_head_stop && !o->no_detector) off = align_up(off + (size_t)n_groups * max_chunks * g * 8 * 4);
    // one group's records are addressed with 32-bit byte offsets
    if ((int64_t)max_chunks * 2 * p->record_floats * 4 > INT32_MAX) return ART_ERR_UNSUPPORTED;
    w.total = off;
    return ART_OK;
}

// Host checks of a decode call and its plan (everything but the workspace).
art_status check_decode_call(const art_decode_shape* shape, const art_decode_opts* opts,
                             const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* page_table, const int32_t* seq_lens,
                             const int32_t* block_list, const int32_t* block_list_len,
                             const void* out, const float* lse, const int32_t* stop_block,
                             Plan* plan) {
    art_status st = make_plan(shape, opts, plan);
    if (st != ART_OK) return st;
    if (shape->batch == 0) return ART_OK;
    if (!q || !k_cache || !v_cache || !page_table || !seq_lens || !out || !lse || !stop_block)
        return ART_ERR_INVALID_ARG;
    if ((block_list == nullptr) != (block_list_len == nullptr)) return ART_ERR_INVALID_ARG;
    if (block_list && shape->max_blocks_per_list <= 0) return ART_ERR_INVALID_ARG;
    if (((uintptr_t)q | (uintptr_t)k_cache | (uintptr_t)v_cache | (uintptr_t)out) % 16)
        return ART_ERR_UNSUPPORTED;
    return ART_OK;
}

// Kernel parameters of a checked call over the workspace at `workspace`,
// then the launch.
art_status enqueue_decode(const Plan& plan, const art_decode_shape* shape,
                          const art_decode_opts* opts, const void* q, const void* k_cache,
                          const void* v_cache, const int32_t* page_table,
                          const int32_t* seq_lens, const int32_t* block_list,
                          const int32_t* block_list_len, void* out, float* lse,
                          int32_t* stop_block, void* workspace, hipStream_t stream) {
    KernelParams k;
    memset(&k, 0, sizeof k);
    k.batch = shape->batch;
    k.num_q_heads = shape->num_q_heads;
    k.num_kv_heads = shape->num_kv_heads;
    k.block_size = shape->block_size;
    k.page_shift = ilog2(shape->page_size);
    k.num_pages = shape->num_pages;
    k.max_pages = shape->max_pages_per_seq;
    k.max_list = shape->max_blocks_per_list;
    k.list_per_head = shape->list_per_head;
    k.ks_page = shape->k_stride_page;
    k.ks_head = shape->k_stride_head;
    k.ks_tok = shape->k_stride_token;
    k.vs_page = shape->v_stride_page;
    k.vs_head = shape->v_stride_head;
    k.vs_tok = shape->v_stride_token;
    k.scale_log2 = (float)((double)opts->softmax_scale * 1.4426950408889634);
    k.tau = opts->tau;
    k.phi = opts->phi;
    k.patience = opts->patience;
    k.probe_stride = opts->probe_stride > 1 ? opts->probe_stride : 1;
    k.scale_of_accumulator = opts->scale_of_accumulator;
    k.no_detector = opts->no_detector;
    k.per_head = opts->per_head_stop && !opts->no_detector;
    k.dense_order = opts->dense_order;
    k.out_bf16 = opts->out_dtype == ART_OUT_BF16;
    k.tiles_per_block = plan.tiles_per_block;
    k.chunk_blocks = plan.chunk_blocks;
    k.max_chunks = plan.max_chunks;
    k.lead_chunks = plan.lead_chunks;
    k.lead_blocks = plan.lead_blocks;
    k.t_cap = plan.t_cap;
    k.n_slots = plan.slots;
    {
        // the work list covers the longest traversal this call can have
        const int64_t cap_tokens = (int64_t)shape->max_pages_per_seq * shape->page_size;
        int64_t t_eff = block_list ? shape->max_blocks_per_list
                                   : (cap_tokens + shape->block_size - 1) / shape->block_size;
        if (t_eff > plan.t_cap) t_eff = plan.t_cap;
        if (t_eff < 1) t_eff = 1;
        k.work_chunks = (int32_t)chunks_for(t_eff, plan.chunk_blocks, plan.lead_chunks, plan.lead_blocks);
    }
    k.record_floats = plan.record_floats;
    k.chunk_recs_lds = plan.chunk_blocks;
    k.loader_partials = plan.loader_partials;
    k.v_in_record = plan.v_in_record;
    k.q = static_cast<const uint16_t*>(q);
    k.k = static_cast<const uint16_t*>(k_cache);
    k.v = static_cast<const uint16_t*>(v_cache);
    k.page_table = page_table;
    k.seq_lens = seq_lens;
    k.block_list = block_list;
    k.block_list_len = block_list_len;
    k.out = out;
    k.lse = lse;
    k.stop_block = stop_block;
    char* ws = static_cast<char*>(workspace);
    k.error_word = reinterpret_cast<uint64_t*>(ws + plan.ws.error_off);
    k.queue = reinterpret_cast<uint64_t*>(ws + plan.ws.queue_off);
    k.stop_word = reinterpret_cast<uint64_t*>(ws + plan.ws.stop_off);
    k.flags = reinterpret_cast<uint64_t*>(ws + plan.ws.flags_off);
    k.records = reinterpret_cast<float*>(ws + plan.ws.records_off);
    k.head_area = reinterpret_cast<int32_t*>(ws + plan.ws.head_off);
    k.epoch = next_epoch();
    k.spin_limit = opts->max_wait_polls > 0 ? (uint32_t)opts->max_wait_polls : kSpinLimit;
    k.max_ahead = opts->max_ahead_chunks;
    if (k.epoch >= (uint64_t(1) << 40)) return ART_ERR_UNSUPPORTED;
    return art::launch_decode(plan, k, stream) == (int)hipSuccess ? ART_OK : ART_ERR_HIP;
}

}  // namespace

extern "C" {

int32_t art_abi_version(void) { return ART_ABI_VERSION; }

const char* art_status_str(int32_t status) {
    switch (status) {
        case ART_OK: return "ART_OK";
        case ART_ERR_INVALID_ARG: return "ART_ERR_INVALID_ARG";
        case ART_ERR_UNSUPPORTED: return "ART_ERR_UNSUPPORTED";
        case ART_ERR_WORKSPACE_TOO_SMALL: return "ART_ERR_WORKSPACE_TOO_SMALL";
        case ART_ERR_HIP: return "ART_ERR_HIP";
        case ART_ERR_BAD_INDEX: return "ART_ERR_BAD_INDEX";
        case ART_ERR_DEVICE_TIMEOUT: return "ART_ERR_DEVICE_TIMEOUT";
        default: return "ART_ERR_UNKNOWN";
    }
}

size_t art_decode_workspace_bytes(const art_decode_shape* shape, const art_decode_opts* opts,
                                  int32_t* status) {
    Plan p;
    art_status st = make_plan(shape, opts, &p);
    if (status) *status = st;
    return st == ART_OK ? p.ws.total : 0;
}

art_status art_workspace_init(void* workspace, size_t bytes, hipStream_t stream) {
    if (!workspace && bytes) return ART_ERR_INVALID_ARG;
    if (bytes % 4) return ART_ERR_INVALID_ARG;
    return art::launch_fill_zero(workspace, bytes, stream) == (int)hipSuccess ? ART_OK : ART_ERR_HIP;
}


art_status art_decode_attention(const art_decode_shape* shape, const art_decode_opts* opts,
                                const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* page_table, const int32_t* seq_lens,
                                const int32_t* block_list, const int32_t* block_list_len,
                                void* out, float* lse, int32_t* stop_block,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
    Plan plan;
    art_status st = check_decode_call(shape, opts, q, k_cache, v_cache, page_table, seq_lens,
                                      block_list, block_list_len, out, lse, stop_block, &plan);
    if (st != ART_OK || shape->batch == 0) return st;
    if (!workspace || workspace_bytes < plan.ws.total) return ART_ERR_WORKSPACE_TOO_SMALL;
    if ((uintptr_t)workspace % 8) return ART_ERR_INVALID_ARG;
    return enqueue_decode(plan, shape, opts, q, k_cache, v_cache, page_table, seq_lens,
                          block_list, block_list_len, out, lse, stop_block, workspace, stream);
}

art_status art_decode_attention_static(const art_decode_shape* shape, const art_decode_opts* opts,
                                       const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* page_table, const int32_t* seq_lens,
                                       const int32_t* block_list, const int32_t* block_list_len,
                                       void* out, float* lse, int32_t* stop_block,
                                       hipStream_t stream) {
    Plan plan;
    art_status st = check_decode_call(shape, opts, q, k_cache, v_cache, page_table, seq_lens,
                                      block_list, block_list_len, out, lse, stop_block, &plan);
    if (st != ART_OK || shape->batch == 0) return st;
    if (plan.ws.total > ART_STATIC_SCRATCH_BYTES) return ART_ERR_WORKSPACE_TOO_SMALL;
    void* scratch = nullptr;
    if (art::static_scratch(stream, &scratch) != (int)hipSuccess) return ART_ERR_HIP;
    return enqueue_decode(plan, shape, opts, q, k_cache, v_cache, page_table, seq_lens,
                          block_list, block_list_len, out, lse, stop_block, scratch, stream);
}

art_status art_validate_inputs(const art_decode_shape* shape, const art_decode_opts* opts,
                               const int32_t* page_table, const int32_t* seq_lens,
                               const int32_t* block_list, const int32_t* block_list_len,
                               hipStream_t stream, int64_t* bad_index, int32_t* bad_where) {
    if (bad_index) *bad_index = -1;
    if (bad_where) *bad_where = -1;
    art_status st = check_shape(shape, opts);
    if (st != ART_OK) return st;
    const int B = shape->batch;
    if (B == 0) return ART_OK;
    if (!page_table || !seq_lens || ((block_list == nullptr) != (block_list_len == nullptr)))
        return ART_ERR_INVALID_ARG;
    const int rows = shape->list_per_head ? shape->num_kv_heads : 1;
    std::vector<int32_t> sl(B), pt((size_t)B * shape->max_pages_per_seq), bll, bl;
    if (hipMemcpyAsync(sl.data(), seq_lens, sizeof(int32_t) * B, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipMemcpyAsync(pt.data(), page_table, sizeof(int32_t) * pt.size(), hipMemcpyDeviceToHost, stream) != hipSuccess)
        return ART_ERR_HIP;
    if (block_list) {
        bll.resize((size_t)B * rows);
        bl.resize((size_t)B * rows * shape->max_blocks_per_list);
        if (hipMemcpyAsync(bll.data(), block_list_len, sizeof(int32_t) * bll.size(), hipMemcpyDeviceToHost, stream) != hipSuccess ||
            (!bl.empty() && hipMemcpyAsync(bl.data(), block_list, sizeof(int32_t) * bl.size(), hipMemcpyDeviceToHost, stream) != hipSuccess))
            return ART_ERR_HIP;
    }
    if (hipStreamSynchronize(stream) != hipSuccess) return ART_ERR_HIP;
    auto fail = [&](int64_t idx, int32_t where) {
        if (bad_index) *bad_index = idx;
        if (bad_where) *bad_where = where;
        return ART_ERR_BAD_INDEX;
    };
    const int64_t cap = (int64_t)shape->max_pages_per_seq * shape->page_size;
    for (int b = 0; b < B; ++b)
        if (sl[b] < 0 || sl[b] > cap) return fail(b, 0);
    for (int b = 0; b < B; ++b) {
        const int64_t npg = ((int64_t)sl[b] + shape->page_size - 1) / shape->page_size;
        for (int64_t i = 0; i < npg; ++i) {
            const int32_t pg = pt[(size_t)b * shape->max_pages_per_seq + i];
            if (pg < 0 || pg >= shape->num_pages) return fail((int64_t)b * shape->max_pages_per_seq + i, 1);
        }
    }
    if (block_list) {
        std::vector<uint8_t> seen;
        for (int b = 0; b < B; ++b) {
            const int64_t nblk = ((int64_t)sl[b] + shape->block_size - 1) / shape->block_size;
            for (int r = 0; r < rows; ++r) {
                const int64_t row = (int64_t)b * rows + r;
                const int32_t n = bll[row];
                if (n < 0 || n > shape->max_blocks_per_list) return fail(row, 3);
                seen.assign((size_t)(nblk > 0 ? nblk : 1), 0);
                for (int32_t i = 0; i < n; ++i) {
                    const int64_t idx = row * shape->max_blocks_per_list + i;
                    const int32_t id = bl[idx];
                    if (id < 0 || id >= nblk || seen[id]) return fail(idx, 2);
                    seen[id] = 1;
                }
            }
        }
    }
    return ART_OK;
}

art_status art_workspace_status(const void* workspace, size_t workspace_bytes, hipStream_t stream,
                                int32_t* device_status) {
    if (!workspace || workspace_bytes < 8 || !device_status) return ART_ERR_INVALID_ARG;
    uint64_t word = 0;
    if (hipStreamSynchronize(stream) != hipSuccess) return ART_ERR_HIP;
    if (hipMemcpy(&word, workspace, 8, hipMemcpyDeviceToHost) != hipSuccess) return ART_ERR_HIP;
    *device_status = word == 0 ? ART_OK : ART_ERR_DEVICE_TIMEOUT;
    return ART_OK;
}

}  // extern "C"

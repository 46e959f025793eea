// ART decode attention kernels for gfx950 (MI355X).
//
// One launch computes, for every (sequence b, KV head kvh) group, the
// block-streaming softmax attention of Sec. 3.1 over the group's traversal
// (recency-first, forward, or a supplied block list, Sec. 3.4), the
// magnitude/direction stability test of Sec. 3.2 (Eq. 2) after every block,
// the patience counter of Eq. (3) and the early break of Algorithm 1.
//
// Work decomposition
//   A group's traversal of T blocks is cut into chunks of consecutive
//   blocks (with the default plan, four leading chunks of 3 blocks, then
//   chunks of C).  The chunks of all groups form eight chunk-major work lists
//   (list x holds the groups 8r + (x + r) mod 8 of every full run r of eight
//   groups, and the leftover groups g with g mod 8 = x: chunk 0 of each, then
//   chunk 1, ...).  The grid is persistent (as many workgroups as the chip holds);
//   workgroups take list indices from epoch-tagged queue words, so
//   workgroups freed by groups that stopped early move on to the groups that
//   stop late.  Each list is handed out in order and a chunk only waits on
//   earlier chunks of its own group, so every wait targets a chunk that some
//   workgroup already holds: no deadlock whatever the dispatch order.
//
//   Loaders (wavefronts 1..3): the leader claims a chunk when one of the two
//   LDS chunk buffers is free; the loaders stream its 64-token tiles from HBM
//   (16-byte loads, four 64-byte row segments per K load instruction, four
//   256-byte rows per V load instruction), compute the scores of all g query
//   heads with v_mfma_f32_16x16x32_bf16 (tokens are the M rows, query heads
//   the N columns, head dims the reduction), the tile softmax in base 2, and
//   P.V on the same MFMA with P split into three bf16 parts (fp32 accuracy),
//   and leave (m, l, sum p v) for each block in LDS.  Chunks after an
//   announced stop are not loaded, and a loader gives up a chunk mid-way
//   once a stop before it is announced.
//
//   Resolver (wavefront 0), per ready chunk:
//     - folds the loaders' partials into the chunk aggregate;
//     - obtains the softmax state after the previous chunk (that chunk's
//       inclusive state, or the nearest inclusive state found by looking
//       back with the aggregates after it folded forward: always the same
//       left fold, so results never depend on timing) and publishes its own
//       inclusive state at once;
//     - replays its blocks from that prefix, running the stability test per
//       block (normalised running output o(t), increment d = o(t) - o(t-1),
//       d_scale = |d|, d_direction = 1 - cos from |o|^2, |d|^2 and o.d
//       without cancellation);
//     - publishes a stability summary, and announces "stop at or before this
//       chunk" at once when the chunk's own blocks hold a run of p stable
//       steps; if the chunk can hold the stop (or is the group's last chunk)
//       it looks back the same way over the stability states (entering
//       patience run, stop already found) and either stops inside the chunk
//       (announces the stop, then writes out/lse/stop_block) or, as the last
//       chunk, writes the untruncated result.
//   Cross-workgroup data goes through the workspace with device-coherent
//   accesses only, as the XCDs of MI355X have separate L2 caches (see the
//   workspace helpers below).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "art_internal.h"

namespace art {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_inff();
constexpr int kD = kHeadDim;

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;  // NaN
  u += 0x7fffu + ((u >> 16) & 1u);                       // round to nearest even
  return u >> 16;
}

// ---- wavefront reductions over the 16 lanes of a DPP row -------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141; // lane i <- lane 7-i within each 8
constexpr int kRowMirror = 0x140;     // lane i <- lane 15-i within each 16

// Every lane of the row ends with the same bits (each step adds the same two
// partial sums, only in swapped operand order).
__device__ __forceinline__ float row_sum(float x) {
  x = x + dpp_f<kQuadXor1>(x);
  x = x + dpp_f<kQuadXor2>(x);
  x = x + dpp_f<kRowHalfMirror>(x);
  x = x + dpp_f<kRowMirror>(x);
  return x;
}
__device__ __forceinline__ float row_max(float x) {
  x = fmaxf(x, dpp_f<kQuadXor1>(x));
  x = fmaxf(x, dpp_f<kQuadXor2>(x));
  x = fmaxf(x, dpp_f<kRowHalfMirror>(x));
  x = fmaxf(x, dpp_f<kRowMirror>(x));
  return x;
}

// LDS written by some lanes of this wave, read by others.  LDS operations of
// one wavefront complete in order; this waits for them and keeps the
// compiler from moving memory operations across.
__device__ __forceinline__ void wave_lds_sync() {
  __asm__ __volatile__("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  __asm__ __volatile__("" ::: "memory");
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// single hardware instructions (about 1 ulp): the same bits wherever used
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fast_sqrt(float x) { return __builtin_amdgcn_sqrtf(x); }

// ---- workspace: cross-workgroup data ---------------------------------------
// Everything one workgroup hands to another (flags, softmax records,
// stability records, the stop announcement) is written and read only with
// agent-scope atomic accesses, which gfx950 performs coherently across the
// XCDs' L2 caches (sc1).  A writer waits for its data stores to complete
// (s_waitcnt vmcnt(0)) before it stores the flag; a reader issues its data
// loads only after the flag load has returned the expected value.  No L2
// write-back or invalidate is needed, so publishing costs a few stores.
__device__ __forceinline__ uint64_t ld_relaxed(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_relaxed32(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_coh_i32(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_i32(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coh_f32(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_f32(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// two adjacent floats through one 64-bit coherent access
__device__ __forceinline__ void ld_coh_f32x2(const float* p, float& a, float& b) {
  const uint64_t w = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  a = __uint_as_float((uint32_t)w);
  b = __uint_as_float((uint32_t)(w >> 32));
}
__device__ __forceinline__ void st_coh_f32x2(float* p, float a, float b) {
  const uint64_t w = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// wait until this wave's global stores have completed; also a compiler
// barrier for memory operations
__device__ __forceinline__ void stores_complete() {
  __asm__ __volatile__("s_waitcnt vmcnt(0)" ::: "memory");
}
__device__ __forceinline__ void compiler_fence() { __asm__ __volatile__("" ::: "memory"); }

// Flag words: epoch << 24 | state << 20 | payload (20 bits).  The stability
// states carry their data in the payload, so that they are published with a
// single store and read with the flag itself.
__device__ __forceinline__ uint64_t make_flag(uint64_t epoch, uint32_t state, uint32_t payload) {
  return (epoch << 24) | ((uint64_t)state << 20) | (uint64_t)payload;
}
__device__ __forceinline__ uint32_t flag_state(uint64_t v, uint64_t epoch) {
  return (v >> 24) == epoch ? (uint32_t)((v >> 20) & 7u) : 0u;
}
__device__ __forceinline__ uint32_t flag_payload(uint64_t v) { return (uint32_t)(v & 0xfffffu); }

// Bounded waits.  A wave that polls spin_limit times without seeing what it
// waits for gives up: it stores this call's epoch and the timeout status in
// the error word and ends.  Every other wait of the launch reads the error
// word every kErrPollEvery polls and ends as soon as it carries this call's
// epoch, so one give-up drains the whole grid within a few polls per wave
// instead of each dependent wait spinning out its own limit.  (A word left
// by an earlier call carries another epoch: it is reported by the status
// call but does not end this one.)
constexpr uint32_t kTimeoutStatus = 6u;   // ART_ERR_DEVICE_TIMEOUT
constexpr uint32_t kErrPollEvery = 16u;
template <typename Params>
__device__ __forceinline__ void raise_timeout(const Params& P) {
  __hip_atomic_store(P.error_word, (P.epoch << 8) | kTimeoutStatus, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
template <typename Params>
__device__ __forceinline__ bool launch_failed(const Params& P) {
  return (ld_relaxed(P.error_word) >> 8) == P.epoch;
}
// Race stress (the build with ART_RACE_STRESS defined, a test build only):
// a pseudo-random delay of up to 7 sleeps of 8128 cycles at every point
// where one workgroup hands data to another or acts on what another handed
// over, keyed by the call, the group, the chunk and the site, so that the
// look-back's producers and consumers meet in orders a plain run rarely
// shows.  Delays only stretch time: every wait stays bounded.
template <typename Params>
__device__ __forceinline__ void stress_delay(const Params& P, int gidx, int k, int site) {
#ifdef ART_RACE_STRESS
  uint32_t h = (uint32_t)P.epoch * 0x9E3779B1u ^ (uint32_t)gidx * 0x85EBCA77u ^
               (uint32_t)k * 0xC2B2AE3Du ^ (uint32_t)site * 0x27D4EB2Fu;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  const uint32_t n = __builtin_amdgcn_readfirstlane((h >> 8) & 7u);
  for (uint32_t i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(127);
#else
  (void)P; (void)gidx; (void)k; (void)site;
#endif
}

// The give-up test of one poll of a wait loop (spin counts the polls made).
template <typename Params>
__device__ __forceinline__ bool wait_expired(const Params& P, uint32_t spin) {
  if (spin >= P.spin_limit) {
    raise_timeout(P);
    return true;
  }
  return (spin % kErrPollEvery) == kErrPollEvery - 1 && launch_failed(P);
}

template <int G>
struct Cfg {
  static constexpr int HPL = G >= 4 ? G / 4 : 1;   // head slots per lane (state layout)
  static constexpr int HC = G > 8 ? 8 : G;          // heads per P.V pass
  static constexpr int REC = G * kD + 2 * G;        // floats per LDS tile record
};

// Per-head softmax state in the "state layout": lane l covers dims
// 8*(l&15) .. +7 of heads (l>>4) + 4*k, k < HPL.  m is in base 2
// (scores * scale * log2 e), L is the mass sum 2^(s - m), o the normalised
// output.  L == 0 is the empty state.
template <int G>
struct State {
  float m[Cfg<G>::HPL];
  float L[Cfg<G>::HPL];
  float o[Cfg<G>::HPL][8];
};

template <int G>
__device__ __forceinline__ void state_clear(State<G>& s) {
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    s.m[k] = kNegInf;
    s.L[k] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s.o[k][e] = 0.f;
  }
}

template <int G>
__device__ __forceinline__ bool slot_valid(int lane, int k) {
  return ((lane >> 4) + 4 * k) < G;
}

// s <- s (+) p : softmax-weighted merge of two disjoint token sets.
// o_new = o + w (o_p - o) with w = mass_p / (mass_s + mass_p) (the increment
// form of Appendix A).  Written with explicit operations so that every call
// site produces the same bits.  Optionally returns the increment d.
template <int G, bool WANT_DELTA>
__device__ __forceinline__ void merge(State<G>& s, const State<G>& p,
                                      float (*delta)[8] = nullptr) {
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    const bool v1 = s.L[k] > 0.f;
    const bool v2 = p.L[k] > 0.f;
    const float mn = v1 ? (v2 ? fmaxf(s.m[k], p.m[k]) : s.m[k]) : p.m[k];
    const float a = v1 ? __fmul_rn(s.L[k], fast_exp2(__fsub_rn(s.m[k], mn))) : 0.f;
    const float bb = v2 ? __fmul_rn(p.L[k], fast_exp2(__fsub_rn(p.m[k], mn))) : 0.f;
    const float Ln = __fadd_rn(a, bb);
    const float w = v2 ? (v1 ? __fmul_rn(bb, fast_rcp(Ln)) : 1.f) : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float d = __fmul_rn(w, __fsub_rn(p.o[k][e], s.o[k][e]));
      if (WANT_DELTA) delta[k][e] = d;
      s.o[k][e] = __fadd_rn(s.o[k][e], d);
    }
    s.m[k] = (v1 || v2) ? mn : kNegInf;
    s.L[k] = Ln;
  }
}

// ---- records: workspace (coherent, normalised) and LDS tiles --------------
// Record layout: o[G][128] | m[G] | L[G].
template <int G>
__device__ __forceinline__ void write_state(float* rec, const State<G>& s, int lane) {
  const int c = lane & 15, r = lane >> 4;
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    const int h = r + 4 * k;
    if (h < G) {
      f32x4* dst = reinterpret_cast<f32x4*>(rec + h * kD + c * 8);
      dst[0] = f32x4{s.o[k][0], s.o[k][1], s.o[k][2], s.o[k][3]};
      dst[1] = f32x4{s.o[k][4], s.o[k][5], s.o[k][6], s.o[k][7]};
      if (c == 0) {
        rec[G * kD + h] = s.m[k];
        rec[G * kD + G + h] = s.L[k];
      }
    }
  }
}

template <int G>
__device__ __forceinline__ void read_state(const float* rec, State<G>& s, int lane) {
  const int c = lane & 15, r = lane >> 4;
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    int h = r + 4 * k;
    if (h >= G) h = 0;  // idle slot: read something valid, never used
    const f32x4* src = reinterpret_cast<const f32x4*>(rec + h * kD + c * 8);
    const f32x4 x0 = src[0], x1 = src[1];
    s.o[k][0] = x0[0]; s.o[k][1] = x0[1]; s.o[k][2] = x0[2]; s.o[k][3] = x0[3];
    s.o[k][4] = x1[0]; s.o[k][5] = x1[1]; s.o[k][6] = x1[2]; s.o[k][7] = x1[3];
    s.m[k] = rec[G * kD + h];
    s.L[k] = rec[G * kD + G + h];
  }
}

// Workspace records go through a buffer resource over the group's record
// area with the sc1 cache policy: agent-coherent 16-byte accesses whose
// completion the compiler tracks like any other load or store.
constexpr int kCoherent = 16;  // buffer cache policy: sc1
constexpr int kLookFirstPasses = 5;  // look-back passes before a chunk publishes its aggregate

__device__ __forceinline__ __amdgpu_buffer_rsrc_t record_rsrc(const KernelParams& P, int gidx) {
  const float* base = P.records + (int64_t)gidx * P.max_chunks * 2 * P.record_floats;
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0,
                                           P.max_chunks * 2 * P.record_floats * 4, 0x00020000);
}

// Layout of a workspace record (G*kD + 2G floats).  Head h's outputs fill
// floats h*kD .. h*kD + 127, first the first halves of the sixteen lanes'
// eight coordinates (lane c: dims 8c .. 8c+3 at 4c), then the second halves
// (dims 8c+4 .. 8c+7 at 64 + 4c), so that each store instruction covers
// whole 64-byte segments (256 contiguous bytes per head) and each segment
// leaves the L2 once, not once per half; m and L of head h follow at G*kD + h
// and G*kD + G + h.
template <int G>
__device__ __forceinline__ void publish_state(__amdgpu_buffer_rsrc_t rs, int rec_off, const State<G>& s,
                                              int lane) {
  const int c = lane & 15, r = lane >> 4;
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    const int h = r + 4 * k;
    if (h < G) {
      const int off = (rec_off + h * kD + c * 4) * 4;
      __builtin_amdgcn_raw_buffer_store_b128(f32x4{s.o[k][0], s.o[k][1], s.o[k][2], s.o[k][3]}, rs, off, 0, kCoherent);
      __builtin_amdgcn_raw_buffer_store_b128(f32x4{s.o[k][4], s.o[k][5], s.o[k][6], s.o[k][7]}, rs, off + 256, 0, kCoherent);
      if (c == 0) {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s.m[k]), rs, (rec_off + G * kD + h) * 4, 0, kCoherent);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s.L[k]), rs, (rec_off + G * kD + G + h) * 4, 0, kCoherent);
      }
    }
  }
}

template <int G>
__device__ __forceinline__ void fetch_state(__amdgpu_buffer_rsrc_t rs, int rec_off, State<G>& s, int lane) {
  const int c = lane & 15, r = lane >> 4;
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    int h = r + 4 * k;
    if (h >= G) h = 0;
    const int off = (rec_off + h * kD + c * 4) * 4;
    const f32x4 x0 = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kCoherent);
    const f32x4 x1 = __builtin_amdgcn_raw_buffer_load_b128(rs, off + 256, 0, kCoherent);
    s.o[k][0] = x0[0]; s.o[k][1] = x0[1]; s.o[k][2] = x0[2]; s.o[k][3] = x0[3];
    s.o[k][4] = x1[0]; s.o[k][5] = x1[1]; s.o[k][6] = x1[2]; s.o[k][7] = x1[3];
    s.m[k] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, (rec_off + G * kD + h) * 4, 0, kCoherent));
    s.L[k] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, (rec_off + G * kD + G + h) * 4, 0, kCoherent));
  }
}

// An LDS block record holds the block's normalised output (the loaders
// normalise it when they write it), its running max and its mass.
template <int G>
__device__ __forceinline__ void read_tile(const float* rec, State<G>& s, int lane) {
  read_state<G>(rec, s, lane);
}

// ---- phase 1: one 64-token tile on one wavefront ---------------------------
template <int G>
__device__ __forceinline__ void load_q(const KernelParams& P, int b, int kvh, int lane, bf16x8 (&qa)[4]) {
  const int h = lane & 15;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (h < G) {
      const uint16_t* src = P.q + ((int64_t)b * P.num_q_heads + kvh * G + h) * kD + (4 * s + (lane >> 4)) * 8;
      const u32x4 w = *reinterpret_cast<const u32x4*>(src);
      qa[s] = __builtin_bit_cast(bf16x8, w);
    } else {
      qa[s] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }
  }
}

__device__ __forceinline__ int clamp_page(const KernelParams& P, int b, int tok) {
  int pg = P.page_table[(int64_t)b * P.max_pages + (tok >> P.page_shift)];
  pg = pg < 0 ? 0 : pg;
  return pg >= P.num_pages ? P.num_pages - 1 : pg;
}

// A 64-token tile on one wavefront.  Both contractions run on
// v_mfma_f32_16x16x32_bf16:
//   - scores transposed, S^T = K Q^T (tokens are the M rows, the query
//     heads of the group the N columns, head dims the reduction), so that
//     each lane ends up holding the probabilities of one head for exactly
//     the eight tokens that the P.V A-operand needs from it;
//   - P.V with P as A (heads x 32 tokens) and V as B (32 tokens x 16 dims).
//     V reaches the B layout (eight tokens of one dim per lane) through LDS,
//     written row-major and read back with ds_read_b64_tr_b16: for groups
//     of up to 4 heads, half tiles through the loader's own staging buffer;
//     for 8 or more, quarter tiles (16 tokens, 4 KiB), through the output
//     part of the very record the tile is about to write when every block
//     is one tile (nothing reads it before the record is written, and the
//     LDS so saved holds longer chunks), else through a 4 KiB staging
//     buffer.  P is split into three bf16 parts (hi + mid + lo carries 24
//     significant bits), so P.V keeps fp32 precision.
// The record written to LDS holds the normalised block output
// sum_j p_hj v_j / l_h [G][128], m_h [G] (base 2) and l_h [G].  pg[n] is the
// (uniform) physical page of 16-token group n.
typedef short v4i16 __attribute__((ext_vector_type(4)));
constexpr int kVPitch = 144;                  // u16 per row of a staging buffer (288 B)
constexpr int kVBufU16 = 32 * kVPitch;        // one half tile: 32 rows
constexpr int kVRow = 128;                    // u16 per row of a quarter-tile stage (256 B)
// Quarter-tile stage: row r's 16-byte piece j sits at piece j ^ 2(r & 3),
// so that the four rows one transposing read touches fall on distinct banks
// (a half-tile buffer pads its rows to 288 bytes for the same end).
__device__ __forceinline__ int vstage_off(int row, int piece) {
  return row * kVRow + ((piece ^ (2 * (row & 3))) << 3);
}

// The first tile of a block writes the block record; each later tile of
// the block (accumulate) is folded into it: both parts rescaled to the
// larger running max and the combined mass, in tile order.
template <int G>
__device__ void compute_tile(const KernelParams& P, int kvh, int L, int tok0, const int (&pg)[4],
                             const bf16x8 (&qa)[4], uint16_t* __restrict__ vbuf,
                             float* __restrict__ rec, bool accumulate) {
  const int lane = threadIdx.x & 63;
  const int lo = lane & 15, g = lane >> 4;
  const int psz_mask = (1 << P.page_shift) - 1;

  if (tok0 >= L) {  // tile past the sequence end: empty partial
    if (accumulate) return;
    for (int i = lane; i < G * kD; i += 64) rec[i] = 0.f;
    if (lane < G) {
      rec[G * kD + lane] = kNegInf;
      rec[G * kD + G + lane] = 0.f;
    }
    return;
  }

  // K: for 16-token group n, lane holds token 16n + lo, dims 32s + 8g .. +7.
  // A 16-aligned group never straddles a page (page_size >= 16, power of
  // two); tokens past L are redirected to token L-1, which lies in the same
  // group or in the last group before it, the group whose page pg[n] then
  // names.
  u32x4 kr[4][4];
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    const int tok = min(tok0 + 16 * n + lo, L - 1);
    const uint16_t* kp = P.k + (int64_t)pg[n] * P.ks_page + (int64_t)kvh * P.ks_head +
                         (int64_t)(tok & psz_mask) * P.ks_tok;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      kr[n][s] = *reinterpret_cast<const u32x4*>(kp + (4 * s + g) * 8);
  }
  // V: lane (lo, g) holds token 4i + g, dims 8lo .. +7; the four tokens of
  // one load instruction are consecutive and lie in group i / 4.  Issued
  // with the K loads so that one memory latency covers the whole tile.
  u32x4 vr[16];
  {
    const uint16_t* vp = P.v + (int64_t)kvh * P.vs_head + lo * 8;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tok = min(tok0 + 4 * i + g, L - 1);
      vr[i] = *reinterpret_cast<const u32x4*>(vp + (int64_t)pg[i >> 2] * P.vs_page +
                                              (int64_t)(tok & psz_mask) * P.vs_tok);
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // S^T[n][r]: token 16n + 4g + r, head lo.
  f32x4 St[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    St[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
      St[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[n][s]), qa[s], St[n], 0, 0, 0);
  }
  // softmax of head lo over the tile: the lane's 16 tokens, then the four
  // lanes lo, lo+16, lo+32, lo+48 (every lane of a column ends with the
  // same bits: max is exact and each step adds the same two values)
  float sc[4][4];
  float mx = kNegInf;
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool ok = (lo < G) && (tok0 + 16 * n + 4 * g + r < L);
      sc[n][r] = ok ? St[n][r] * P.scale_log2 : kNegInf;
      mx = fmaxf(mx, sc[n][r]);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  float ls = 0.f;
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = mx == kNegInf ? 0.f : fast_exp2(sc[n][r] - mx);
      sc[n][r] = p;
      ls += p;
    }
  ls = ls + __shfl_xor(ls, 16);
  ls = ls + __shfl_xor(ls, 32);
  if (g == 0 && lo < G && !accumulate) {
    rec[G * kD + lo] = mx;
    rec[G * kD + G + lo] = ls;
  }

  // A operands of the two 32-token K-steps c: element e of lane (lo, g) is
  // p of head lo at token 16(2c + e/4) + 4g + e%4, in three bf16 parts.
  bf16x8 a[2][3];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    uint32_t w[3][4];
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      uint32_t part[3][2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = 2 * e2 + h;
        const float p = sc[2 * c + (e >> 2)][e & 3];
        const uint32_t b0 = f32_to_bf16_bits(p);
        const float r1 = p - __uint_as_float(b0 << 16);
        const uint32_t b1 = f32_to_bf16_bits(r1);
        const float r2 = r1 - __uint_as_float(b1 << 16);
        part[0][h] = b0;
        part[1][h] = b1;
        part[2][h] = f32_to_bf16_bits(r2);
      }
#pragma unroll
      for (int j = 0; j < 3; ++j) w[j][e2] = part[j][0] | (part[j][1] << 16);
    }
#pragma unroll
    for (int j = 0; j < 3; ++j) a[c][j] = __builtin_bit_cast(bf16x8, u32x4{w[j][0], w[j][1], w[j][2], w[j][3]});
  }

  // P.V over the two halves of the tile.  B for K-step c and dims
  // 16d .. 16d+15: lane (lo, g) needs V[token of element e][16d + lo]; in
  // each 16-lane group, source lane 4k + q of a transposing read points at
  // row 4g + k of a 16-row quarter (then of the next one), columns
  // 16d + 4q .. +3.
  f32x4 acc[8];
#pragma unroll
  for (int d = 0; d < 8; ++d) acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int rk = lo >> 2, cq = lo & 3;
  if constexpr (G >= 8) {
    // a quarter at a time, the first quarter's B parts (elements 0..3) kept
    // in registers until the second's are read
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      v4i16 r0[8];
#pragma unroll
      for (int qh = 0; qh < 2; ++qh) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          *reinterpret_cast<u32x4*>(vbuf + vstage_off(4 * i + g, lo)) = vr[8 * c + 4 * qh + i];
        wave_lds_sync();
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          const v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) v4i16*)(vbuf + vstage_off(4 * g + rk, 2 * d + (cq >> 1)) +
                                                         4 * (cq & 1)));
          if (qh == 0) {
            r0[d] = r;
          } else {
            const bf16x8 b = __builtin_bit_cast(bf16x8, __builtin_shufflevector(r0[d], r, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
            for (int j = 0; j < 3; ++j) acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[c][j], b, acc[d], 0, 0, 0);
          }
        }
        wave_lds_sync();  // the reads of this quarter complete before the next one is written
      }
    }
  } else {
    // a whole half at a time; the row pitch of 288 bytes puts the 16 lanes
    // of a group on 32 distinct banks
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<u32x4*>(vbuf + (4 * i + g) * kVPitch + 8 * lo) = vr[8 * c + i];
      wave_lds_sync();
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        const v4i16 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16*)(vbuf + (4 * g + rk) * kVPitch + 16 * d + 4 * cq));
        const v4i16 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16*)(vbuf + (16 + 4 * g + rk) * kVPitch + 16 * d + 4 * cq));
        const bf16x8 b = __builtin_bit_cast(bf16x8, __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int j = 0; j < 3; ++j) acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[c][j], b, acc[d], 0, 0, 0);
      }
      wave_lds_sync();  // the reads of this half complete before the next half is written
    }
  }
  // acc[d][r]: head 4g + r, dim 16d + lo.  A block's first tile divides
  // its sums by the mass l_h written to the record above; a later tile's
  // fold factors come from row 0 of the lanes (g = 0, head lo) through the
  // staging buffer, which the P.V loop no longer reads (a record never
  // stages its own later tiles: records stage only blocks of one tile).
  if (!accumulate) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * g + r;
      if (h < G) {
        const float l = rec[G * kD + G + h];
        const float inv = l > 0.f ? fast_rcp(l) : 0.f;
#pragma unroll
        for (int d = 0; d < 8; ++d) rec[h * kD + 16 * d + lo] = __fmul_rn(acc[d][r], inv);
      }
    }
    return;
  }
  // fold into the block record: o = (o_rec L_rec so + sum_tile sn) / L_new
  float* scale = reinterpret_cast<float*>(vbuf);
  if (g == 0 && lo < G) {
    const float mo = rec[G * kD + lo], lo_sum = rec[G * kD + G + lo];
    const float mn = fmaxf(mo, mx);
    const float so = mo == kNegInf ? 0.f : fast_exp2(mo - mn);
    const float sn = mx == kNegInf ? 0.f : fast_exp2(mx - mn);
    const float a = __fmul_rn(lo_sum, so);
    const float Ln = __fadd_rn(a, __fmul_rn(ls, sn));
    const float inv = Ln > 0.f ? fast_rcp(Ln) : 0.f;
    rec[G * kD + lo] = mn;
    rec[G * kD + G + lo] = Ln;
    scale[lo] = __fmul_rn(a, inv);
    scale[G + lo] = __fmul_rn(sn, inv);
  }
  wave_lds_sync();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = 4 * g + r;
    if (h < G) {
      const float so = scale[h], sn = scale[G + h];
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        float* x = rec + h * kD + 16 * d + lo;
        *x = __fadd_rn(__fmul_rn(*x, so), __fmul_rn(acc[d][r], sn));
      }
    }
  }
  wave_lds_sync();  // the scale factors are read before the buffer is reused
}

// ---- phase 2 helpers ----------------------------------------------------------
// Chunk geometry: the first lead_chunks chunks of a traversal hold
// lead_blocks blocks each, every later one chunk_blocks.
__device__ __forceinline__ int chunk_start(const KernelParams& P, int k) {
  return k < P.lead_chunks ? k * P.lead_blocks
                           : P.lead_chunks * P.lead_blocks + (k - P.lead_chunks) * P.chunk_blocks;
}
__device__ __forceinline__ int chunks_for(const KernelParams& P, int T) {
  const int lead_T = P.lead_chunks * P.lead_blocks;
  return T <= lead_T ? (T + P.lead_blocks - 1) / P.lead_blocks
                     : P.lead_chunks + (T - lead_T + P.chunk_blocks - 1) / P.chunk_blocks;
}

struct StabSummary {   // one chunk's own blocks (entering run taken as 0)
  int32_t lead;        // leading stable blocks
  int32_t trail;       // trailing stable blocks
  int32_t len;         // blocks in the chunk
  int32_t fis;         // first block (0-based) where the chunk's own run reaches p, or -1
};
struct StabState {     // after a prefix of chunks
  int32_t stopped;     // 1 if the stop lies in the prefix
  int32_t stop_t;      // 1-based traversal step of the stop
  int32_t run;         // consecutive stable steps ending the prefix (if not stopped)
  int32_t pad;
};

// Payloads: a summary packs lead, trail, len (each <= 16) and fis + 1 in
// five bits each; a stability state packs `stopped` (bit 19) and the run
// (19 bits; traversals are shorter than 2^19 blocks, so it is exact).
__device__ __forceinline__ uint32_t pack_summary(const StabSummary& y) {
  return (uint32_t)y.lead | ((uint32_t)y.trail << 5) | ((uint32_t)y.len << 10) | ((uint32_t)(y.fis + 1) << 15);
}
__device__ __forceinline__ StabSummary unpack_summary(uint32_t p) {
  return StabSummary{(int32_t)(p & 31u), (int32_t)((p >> 5) & 31u), (int32_t)((p >> 10) & 31u),
                     (int32_t)((p >> 15) & 31u) - 1};
}
__device__ __forceinline__ uint32_t pack_stab(const StabState& x) {
  return ((uint32_t)(x.stopped != 0) << 19) | ((uint32_t)x.run & 0x7ffffu);
}
__device__ __forceinline__ StabState unpack_stab(uint32_t p) {
  return StabState{(int32_t)((p >> 19) & 1u), 0, (int32_t)(p & 0x7ffffu), 0};
}

__device__ __forceinline__ StabState stab_fold(StabState x, StabSummary y, int t0, int patience) {
  if (x.stopped) return x;
  StabState r = x;
  if (y.lead > 0 && (int64_t)x.run + y.lead >= patience) {
    r.stopped = 1;
    r.stop_t = t0 + (patience - x.run - 1) + 1;
  } else if (y.fis >= 0) {
    r.stopped = 1;
    r.stop_t = t0 + y.fis + 1;
  } else {
    r.run = (y.lead == y.len) ? x.run + y.len : y.trail;
  }
  return r;
}

// The stop announcement of a group is one word: epoch << 24 | chunk, where
// the chunk holds the stop or lies after it.  Chunks after the announced one
// are moot: loaders skip them and their resolvers give up.
__device__ __forceinline__ bool stop_word_before(uint64_t v, uint64_t epoch, int me) {
  return (v >> kQueueBits) == epoch && (int)(v & ((1ull << kQueueBits) - 1ull)) < me;
}
__device__ __forceinline__ bool stop_announced_before(const KernelParams& P, int gidx, int me) {
  return stop_word_before(ld_relaxed(P.stop_word + gidx), P.epoch, me);
}
// Lowers the announcement to chunk k unless this call already announced a
// chunk <= k (a word of an earlier call, whatever its bits, is replaced).
// Several chunks of a group may announce; each compare-and-swap that fails
// saw another announcement land, so the loop ends.  Lane 0 only.
__device__ void announce_stop(const KernelParams& P, int gidx, int k) {
  stress_delay(P, gidx, k, 8);
  uint64_t* w = P.stop_word + gidx;
  const uint64_t mine = (P.epoch << kQueueBits) | (uint64_t)k;
  uint64_t cur = ld_relaxed(w);
  for (uint32_t spin = 0; !stop_word_before(cur, P.epoch, k + 1) && spin < P.spin_limit; ++spin)
    if (__hip_atomic_compare_exchange_strong(w, &cur, mine, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      break;
}

// Look-back over the flags of chunks me-1, me-2, ... of group gidx, 64 per
// poll (one per lane): returns the nearest chunk j whose state is >= need_hi
// such that every chunk strictly between j and `me` has state >= need_lo,
// -1 if all chunks 0..me-1 have state >= need_lo and none >= need_hi, or -2
// when a stop in a chunk before `me` has been announced or the spin limit is
// reached (the error word is set then).  Wave-uniform.
__device__ int lookback_scan(const KernelParams& P, int gidx, int me, uint32_t need_lo,
                             uint32_t need_hi, int lane) {
  const uint64_t* flags = P.flags + (int64_t)gidx * P.max_chunks;
  int hi = me - 1;
  uint32_t it = 0;
  while (hi >= 0) {
    const int idx = hi - lane;
    const uint32_t st = idx >= 0 ? flag_state(ld_relaxed(flags + idx), P.epoch) : 0u;
    const uint64_t have_hi = __ballot(idx >= 0 && st >= need_hi);
    const uint64_t have_lo = __ballot(idx < 0 || st >= need_lo);
    const int first = have_hi ? __ffsll((unsigned long long)have_hi) - 1 : 64;
    const uint64_t need = first >= 64 ? ~0ull : ((1ull << first) - 1ull);
    if ((have_lo & need) == need) {
      if (first < 64) return hi - first;
      hi -= 64;  // 64 chunks with aggregates but no inclusive state: look further back
      continue;
    }
    if (stop_announced_before(P, gidx, me)) return -2;
    if (wait_expired(P, ++it)) return -2;
    __builtin_amdgcn_s_sleep(2);
  }
  return -1;
}

// One pass of lookback_scan with no wait: the index found, -1 for an empty
// prefix, or -3 when a chunk in the way has not published yet.
__device__ int lookback_once(const KernelParams& P, int gidx, int me, uint32_t need_lo,
                             uint32_t need_hi, int lane) {
  const uint64_t* flags = P.flags + (int64_t)gidx * P.max_chunks;
  for (int hi = me - 1; hi >= 0; hi -= 64) {
    const int idx = hi - lane;
    const uint32_t st = idx >= 0 ? flag_state(ld_relaxed(flags + idx), P.epoch) : 0u;
    const uint64_t have_hi = __ballot(idx >= 0 && st >= need_hi);
    const uint64_t have_lo = __ballot(idx < 0 || st >= need_lo);
    const int first = have_hi ? __ffsll((unsigned long long)have_hi) - 1 : 64;
    const uint64_t need = first >= 64 ? ~0ull : ((1ull << first) - 1ull);
    if ((have_lo & need) != need) return -3;
    if (first < 64) return hi - first;
  }
  return -1;
}

// Summaries of consecutive chunks compose (entering run 0 throughout):
// A then B has the blocks of both, leads with A's lead (extended by B's if A
// is stable throughout), trails with B's trail (extended by A's if B is),
// and reaches the patience first inside A, else where A's trailing run and
// B's leading run together reach it, else inside B.  Folding a state with
// A then B equals folding it with the composition (the same integers).
__device__ __forceinline__ StabSummary seg_combine(StabSummary a, StabSummary b, int patience) {
  StabSummary r;
  r.len = a.len + b.len;
  r.lead = a.lead == a.len ? a.len + b.lead : a.lead;
  r.trail = b.trail == b.len ? b.len + a.trail : b.trail;
  if (a.fis >= 0) r.fis = a.fis;
  else if (b.lead > 0 && (int64_t)a.trail + b.lead >= patience) r.fis = a.len + (patience - a.trail) - 1;
  else if (b.fis >= 0) r.fis = a.len + b.fis;
  else r.fis = -1;
  return r;
}

// Stability state on entering chunk `me` of group gidx: the nearest chunk j
// before it that published its stability state, folded with the summaries
// of the chunks between (every chunk between must have published its
// summary).  One backward pass, 64 flags per read (lane u holds chunk
// hi - u): each complete window's summaries are composed across the lanes
// in six shuffle steps and put in front of the composition of the later
// windows.  A flag read once at its summary may later show the chunk's own
// state, which is the fold of every chunk up to it, so the summary already
// used gives the same integers.  Returns false when a stop before `me` has
// been announced or the spin limit is reached.
__device__ bool stab_entering(const KernelParams& P, int gidx, int me, StabState& x, int lane) {
  const uint64_t* flags = P.flags + (int64_t)gidx * P.max_chunks;
  StabSummary acc{0, 0, 0, -1};  // composition of the chunks after the window
  int hi = me - 1, j = -1;       // j: the chunk that holds the state, if any
  uint32_t it = 0;
  x = StabState{0, 0, 0, 0};
  while (hi >= 0) {
    const int idx = hi - lane;
    const uint64_t v = idx >= 0 ? ld_relaxed(flags + idx) : 0ull;
    const uint32_t st = idx >= 0 ? flag_state(v, P.epoch) : 0u;
    const uint64_t have_st = __ballot(idx >= 0 && st >= kStabInclusive);
    const uint64_t have_sum = __ballot(idx < 0 || st >= kStabSummary);
    const int first = have_st ? __ffsll((unsigned long long)have_st) - 1 : 64;
    const uint64_t need = first >= 64 ? ~0ull : ((1ull << first) - 1ull);
    if ((have_sum & need) != need) {
      if (stop_announced_before(P, gidx, me)) return false;
      if (wait_expired(P, ++it)) return false;
      __builtin_amdgcn_s_sleep(2);
      continue;
    }
    stress_delay(P, gidx, me, 16);
    // the window's summaries (lanes below `first` that hold a chunk), in
    // chunk order: lane u + d holds the earlier chunk.  Within a window every
    // count is below 2^11, so a summary travels as two words: lead | trail
    // << 16 and len | (fis + 1) << 16.
    const uint32_t pl = flag_payload(v);
    uint32_t w0 = 0u, w1 = 0u;
    if (lane < first && idx >= 0) {
      const StabSummary y = unpack_summary(pl);
      w0 = (uint32_t)y.lead | ((uint32_t)y.trail << 16);
      w1 = (uint32_t)y.len | ((uint32_t)(y.fis + 1) << 16);
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t e0 = __shfl_down(w0, d), e1 = __shfl_down(w1, d);
      if ((lane & (2 * d - 1)) == 0 && lane + d < 64) {
        const StabSummary c = seg_combine(
            StabSummary{(int32_t)(e0 & 0xffffu), (int32_t)(e0 >> 16), (int32_t)(e1 & 0xffffu), (int32_t)(e1 >> 16) - 1},
            StabSummary{(int32_t)(w0 & 0xffffu), (int32_t)(w0 >> 16), (int32_t)(w1 & 0xffffu), (int32_t)(w1 >> 16) - 1},
            P.patience);
        w0 = (uint32_t)c.lead | ((uint32_t)c.trail << 16);
        w1 = (uint32_t)c.len | ((uint32_t)(c.fis + 1) << 16);
      }
    }
    w0 = __builtin_amdgcn_readfirstlane(w0);
    w1 = __builtin_amdgcn_readfirstlane(w1);
    const StabSummary wsum{(int32_t)(w0 & 0xffffu), (int32_t)(w0 >> 16), (int32_t)(w1 & 0xffffu),
                           (int32_t)(w1 >> 16) - 1};
    acc = seg_combine(wsum, acc, P.patience);
    if (first < 64) {
      x = unpack_stab(__builtin_amdgcn_readlane(pl, first));
      j = hi - first;
      break;
    }
    hi -= 64;
  }
  // the summaries after chunk j (after none: from chunk 0 on)
  x = stab_fold(x, acc, chunk_start(P, j + 1), P.patience);
  return true;
}

// States whose data sits in the workspace records: the flag goes out once
// the record stores have completed.
__device__ __forceinline__ void publish(const KernelParams& P, int gidx, int k, uint32_t state, int lane) {
  stress_delay(P, gidx, k, 1);
  stores_complete();
  if (lane == 0)
    __hip_atomic_store(P.flags + (int64_t)gidx * P.max_chunks + k, make_flag(P.epoch, state, 0),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// States carried in the flag word itself: one store, no wait.
__device__ __forceinline__ void publish_word(const KernelParams& P, int gidx, int k, uint32_t state,
                                             uint32_t payload, int lane) {
  stress_delay(P, gidx, k, 2 + (int)state);
  if (lane == 0)
    __hip_atomic_store(P.flags + (int64_t)gidx * P.max_chunks + k, make_flag(P.epoch, state, payload),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <int G>
__device__ void write_outputs(const KernelParams& P, int b, int kvh, const State<G>& s,
                              int stop, int lane, uint32_t heads = 0xffffffffu,
                              bool write_stop = true) {
  const int c = lane & 15, r = lane >> 4;
#pragma unroll
  for (int k = 0; k < Cfg<G>::HPL; ++k) {
    const int h = r + 4 * k;
    if (h >= G || !((heads >> h) & 1u)) continue;
    const int64_t row = (int64_t)b * P.num_q_heads + kvh * G + h;
    if (P.out_bf16) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = f32_to_bf16_bits(s.o[k][2 * e]) | (f32_to_bf16_bits(s.o[k][2 * e + 1]) << 16);
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(P.out) + row * kD + c * 8) = u32x4{w[0], w[1], w[2], w[3]};
    } else {
      f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(P.out) + row * kD + c * 8);
      dst[0] = f32x4{s.o[k][0], s.o[k][1], s.o[k][2], s.o[k][3]};
      dst[1] = f32x4{s.o[k][4], s.o[k][5], s.o[k][6], s.o[k][7]};
    }
    if (c == 0) {
      // natural log of sum exp(scale q.k): (m + log2 L) * ln 2
      P.lse[row] = (s.m[k] + __log2f(s.L[k])) * 0.69314718055994531f;
    }
  }
  if (write_stop && lane == 0) P.stop_block[(int64_t)b * P.num_kv_heads + kvh] = stop;
}

struct GroupInfo {
  int b, kvh, L, nblk, T, n_chunks;
  const int32_t* list;
};

// Traversal of group gidx (indices are clamped: malformed input never makes
// a kernel read outside the arrays the shape describes).
// From the raw sequence length and list length of the group (the list
// length is ignored for dense traversals).
__device__ __forceinline__ GroupInfo group_info_raw(const KernelParams& P, int gidx, int L_raw, int T_raw) {
  GroupInfo g;
  g.b = gidx / P.num_kv_heads;
  g.kvh = gidx - g.b * P.num_kv_heads;
  const int64_t cap = (int64_t)P.max_pages << P.page_shift;
  const int L = L_raw < 0 ? 0 : (int)min((int64_t)L_raw, cap);
  g.L = L;
  g.nblk = (L + P.block_size - 1) / P.block_size;
  g.list = nullptr;
  int T = g.nblk;
  if (P.block_list) {
    const int row = P.list_per_head ? gidx : g.b;
    T = T_raw < 0 ? 0 : min(T_raw, P.max_list);
    g.list = P.block_list + (int64_t)row * P.max_list;
  }
  if (g.nblk == 0) T = 0;
  g.T = min(T, P.t_cap);
  g.n_chunks = chunks_for(P, g.T);
  return g;
}

__device__ __forceinline__ int raw_list_len(const KernelParams& P, int gidx) {
  if (!P.block_list) return 0;
  const int b = gidx / P.num_kv_heads;
  return P.block_list_len[P.list_per_head ? gidx : b];
}

__device__ __forceinline__ GroupInfo group_info(const KernelParams& P, int gidx) {
  return group_info_raw(P, gidx, P.seq_lens[gidx / P.num_kv_heads], raw_list_len(P, gidx));
}

template <int G>
__device__ void write_empty_wave(const KernelParams& P, int b, int kvh, int lane) {
  for (int i = lane; i < G * kD; i += 64) {
    const int64_t idx = ((int64_t)b * P.num_q_heads + kvh * G) * kD + i;
    if (P.out_bf16) static_cast<uint16_t*>(P.out)[idx] = 0;
    else static_cast<float*>(P.out)[idx] = 0.f;
  }
  if (lane < G) P.lse[(int64_t)b * P.num_q_heads + kvh * G + lane] = kNegInf;
  if (P.per_head) {
    if (lane < G) P.stop_block[(int64_t)b * P.num_q_heads + kvh * G + lane] = 0;
  } else if (lane == 0) {
    P.stop_block[(int64_t)b * P.num_kv_heads + kvh] = 0;
  }
}

constexpr int kLoaders = kWaves - 1;   // wavefronts 1..3 stream tiles
constexpr int kMaxSlots = 3;           // chunk buffers in LDS (the plan picks 2 or 3)
constexpr int kLenCache = 256;         // sequence lengths kept in LDS
enum SlotState : int { kSlotFree = 0, kSlotLoading = 1, kSlotReady = 2, kSlotEnd = 3 };
// slot metadata words
constexpr int kMetaSeq = 0, kMetaState = 1, kMetaGroup = 2, kMetaChunk = 3, kMetaDone = 4, kMetaAbort = 5;
constexpr int kMetaLen = 6, kMetaListLen = 7;  // raw seq_len and list length of the group

__device__ __forceinline__ int lds_ld(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_st(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Work queues.  The chunks of the launch form kQueues chunk-major lists:
// queue x holds n_x groups, and its index i stands for chunk i / n_x of
// group x + kQueues * (i % n_x), rotated within its run of kQueues groups
// (see the claim).  Each
// list is handed out from its own workspace word (call epoch << 24 | next
// index) by one fetch-and-add (claim_issue; claim_finish decodes it), so
// that claims spread over kQueues atomic units.  A word left by an earlier
// call is replaced by compare-and-swap with this call's epoch and index 1,
// which hands out index 0; claims that raced with the replacement retry.
// Every chunk a chunk can wait on belongs to the same group, hence to the
// same list, and each list is handed out in increasing order: a chunk only
// ever waits on chunks that some workgroup already holds.  Lane 0 only /
// wave-uniform result.
__device__ __forceinline__ uint64_t* queue_word(const KernelParams& P, int x) {
  return P.queue + (int64_t)x * kQueueStride;
}

__device__ __forceinline__ uint64_t claim_issue(const KernelParams& P, int x, int lane) {
  return lane == 0 ? __hip_atomic_fetch_add(queue_word(P, x), 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                   : 0ull;
}

__device__ int claim_finish(const KernelParams& P, int x, uint64_t v, int lane) {
  int q = 0;
  if (lane == 0) {
    uint64_t* w = queue_word(P, x);
    const uint64_t mask = (1ull << kQueueBits) - 1ull;
    if ((v >> kQueueBits) == P.epoch) {
      q = (int)(v & mask);
    } else {
      uint64_t cur = v + 1ull;
      for (uint32_t spin = 0;; ++spin) {
        if ((cur >> kQueueBits) == P.epoch) {
          v = __hip_atomic_fetch_add(w, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if ((v >> kQueueBits) == P.epoch) {
            q = (int)(v & mask);
            break;
          }
          cur = v + 1ull;
        } else if (__hip_atomic_compare_exchange_strong(w, &cur, (P.epoch << kQueueBits) | 1ull,
                                                        __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT)) {
          q = 0;
          break;
        }
        if (wait_expired(P, spin)) {
          q = 0x7fffffff;
          break;
        }
      }
    }
  }
  return __builtin_amdgcn_readfirstlane(q);
}

// ---- per-query-head termination ---------------------------------------------
// The per-head reading of the test: every query head of a group keeps its
// own patience counter (Eq. 3) and stops on its own; its out and lse are
// those at its own stop (stop_block [batch][num_q_heads] holds each head's
// stop, T for a head that never stops), and the group stops reading blocks
// once its last head has stopped.  The chunk's summaries
// and states of the stability monoid are kept per head in the workspace's
// head area, [chunk][head][8] int32 (lead, trail, len, fis | stopped, run),
// written by lane h for head h and published by the chunk's flag as in the
// group reading.  A summary stays valid after the chunk's state is
// published, so the fold below never meets a changed word.
__device__ __forceinline__ int32_t* head_area(const KernelParams& P, int gidx, int k, int G) {
  return P.head_area + ((int64_t)gidx * P.max_chunks + k) * (int64_t)(G * 8);
}

// The nearest chunk before `me` that published its stability state, such
// that every chunk between published its summary: j >= -1, or -2 when a
// stop before `me` has been announced or a wait gave up.
__device__ int stab_scan(const KernelParams& P, int gidx, int me, int lane) {
  const uint64_t* flags = P.flags + (int64_t)gidx * P.max_chunks;
  int hi = me - 1;
  uint32_t it = 0;
  while (hi >= 0) {
    const int idx = hi - lane;
    const uint32_t st = idx >= 0 ? flag_state(ld_relaxed(flags + idx), P.epoch) : 0u;
    const uint64_t have_st = __ballot(idx >= 0 && st >= kStabInclusive);
    const uint64_t have_sum = __ballot(idx < 0 || st >= kStabSummary);
    const int first = have_st ? __ffsll((unsigned long long)have_st) - 1 : 64;
    const uint64_t need = first >= 64 ? ~0ull : ((1ull << first) - 1ull);
    if ((have_sum & need) == need) {
      if (first < 64) return hi - first;
      hi -= 64;
      continue;
    }
    if (stop_announced_before(P, gidx, me)) return -2;
    if (wait_expired(P, ++it)) return -2;
    __builtin_amdgcn_s_sleep(2);
  }
  return -1;
}

template <int G>
__device__ void resolve_heads(const KernelParams& P, int gidx, int k, const GroupInfo& gi,
                              const float* blocks, const State<G>& pre, uint32_t head_bits,
                              int t0, int nb, int lane) {
  constexpr int REC = Cfg<G>::REC;
  const int n_chunks = gi.n_chunks, T = gi.T;
  const bool mine = lane < G;   // lane h holds head h
  int32_t* my = head_area(P, gidx, k, G) + lane * 8;
  StabSummary sm{0, 0, 0, -1};
  if (mine) {
    int run = 0, lead = 0, fis = -1;
    bool leading = true;
    for (int i = 0; i < nb; ++i) {
      const bool st = (head_bits >> i) & 1u;
      run = st ? run + 1 : 0;
      if (leading) {
        if (st) ++lead;
        else leading = false;
      }
      if (fis < 0 && run >= P.patience) fis = i;
    }
    sm = StabSummary{lead, run, nb, fis};
    st_coh_i32(my + 0, lead);
    st_coh_i32(my + 1, run);
    st_coh_i32(my + 2, nb);
    st_coh_i32(my + 3, fis);
  }
  stores_complete();
  publish_word(P, gidx, k, kStabSummary, 0u, lane);
  // every head reaches its patience inside this chunk: the group's stop lies
  // here or before, whatever the chunks before hold
  const bool all_fis = __all(!mine || sm.fis >= 0);
  if (all_fis && lane == 0) announce_stop(P, gidx, k);
  // no head can stop in a chunk whose first block is unstable for it and
  // whose own runs stay short (the last chunk still writes what is left)
  if (__all(!mine || (sm.lead == 0 && sm.fis < 0)) && k != n_chunks - 1) return;

  // entering state per head: the nearest published state, then the
  // summaries after it
  stress_delay(P, gidx, k, 11);
  const int j = stab_scan(P, gidx, k, lane);
  if (j == -2) return;
  stress_delay(P, gidx, k, 12);
  StabState x{0, 0, 0, 0};
  if (mine && j >= 0) {
    const int32_t* w = head_area(P, gidx, j, G) + lane * 8;
    x.stopped = ld_coh_i32(w + 4);
    x.run = ld_coh_i32(w + 5);
  }
  if (k - (j + 1) <= 4 * G) {
    // a short way back (up to one round trip per head either way): every
    // head folds its own summaries, lane h head h, four chunks' words in
    // flight
    for (int i0 = j + 1; i0 < k; i0 += 4) {
      const int n = min(4, k - i0);
      int32_t v[4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (mine && u < n) {
          const int32_t* w = head_area(P, gidx, i0 + u, G) + lane * 8;
#pragma unroll
          for (int f = 0; f < 4; ++f) v[u][f] = ld_coh_i32(w + f);
        }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (mine && u < n)
          x = stab_fold(x, StabSummary{v[u][0], v[u][1], v[u][2], v[u][3]}, chunk_start(P, i0 + u), P.patience);
    }
  } else {
    // a long way back (the last chunk of a traversal with no stop before):
    // 64 chunks per read (lane u: chunk i0 + u), composed across the lanes
    // for each head in turn
    for (int i0 = j + 1; i0 < k; i0 += 64) {
      const bool in = lane < k - i0;
      const int32_t* wc = head_area(P, gidx, in ? i0 + lane : i0, G);
      const int t_win = chunk_start(P, i0);
      for (int h = 0; h < G; ++h) {
        StabSummary c{0, 0, 0, -1};
        if (in) c = StabSummary{ld_coh_i32(wc + h * 8), ld_coh_i32(wc + h * 8 + 1), ld_coh_i32(wc + h * 8 + 2),
                                ld_coh_i32(wc + h * 8 + 3)};
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const StabSummary e{__shfl_down(c.lead, d), __shfl_down(c.trail, d), __shfl_down(c.len, d),
                              __shfl_down(c.fis, d)};
          if ((lane & (2 * d - 1)) == 0 && lane + d < 64) c = seg_combine(c, e, P.patience);
        }
        const StabSummary comp{__builtin_amdgcn_readfirstlane(c.lead), __builtin_amdgcn_readfirstlane(c.trail),
                               __builtin_amdgcn_readfirstlane(c.len), __builtin_amdgcn_readfirstlane(c.fis)};
        if (lane == h) x = stab_fold(x, comp, t_win, P.patience);
      }
    }
  }
  const StabState y = mine ? stab_fold(x, sm, t0, P.patience) : x;
  if (mine) {
    st_coh_i32(my + 4, y.stopped);
    st_coh_i32(my + 5, y.run);
  }
  stores_complete();
  const bool all_before = __all(!mine || x.stopped);
  const bool all_after = __all(!mine || y.stopped);
  if (!all_before && all_after && !all_fis && lane == 0) announce_stop(P, gidx, k);
  publish_word(P, gidx, k, kStabInclusive, 0u, lane);
  if (all_before) return;   // every head stopped before this chunk

  // heads whose stop lies in this chunk: o(t_h) again from the prefix, by
  // the same merges as the replay
  const int rel = (mine && !x.stopped && y.stopped) ? y.stop_t - t0 - 1 : -1;
  int rel_h[G];
  int last_rel = -1;
  uint32_t never = 0;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    rel_h[h] = __builtin_amdgcn_readlane(rel, h);
    last_rel = max(last_rel, rel_h[h]);
    if (!__builtin_amdgcn_readlane((int)y.stopped, h)) never |= 1u << h;
  }
  int32_t* head_stop = P.stop_block + (int64_t)gi.b * P.num_q_heads + gi.kvh * G;
  if (rel >= 0) head_stop[lane] = y.stop_t;
  // one pass of the replay's merges from the prefix: each head stopping
  // here is written at its block; in the group's last chunk, heads that
  // never stopped get the state after the last block (the whole traversal)
  const bool finish = !all_after && k == n_chunks - 1;
  const int upto = finish ? nb - 1 : last_rel;
  if (upto >= 0) {
    State<G> o = pre, t;
    for (int i = 0; i <= upto; ++i) {
      read_tile<G>(blocks + i * REC, t, lane);
      merge<G, false>(o, t);
      uint32_t here = 0;
#pragma unroll
      for (int h = 0; h < G; ++h)
        if (rel_h[h] == i) here |= 1u << h;
      if (here) write_outputs<G>(P, gi.b, gi.kvh, o, 0, lane, here, false);
    }
    if (finish) {
      write_outputs<G>(P, gi.b, gi.kvh, o, T, lane, never, false);
      if (mine && ((never >> lane) & 1u)) head_stop[lane] = T;
    }
  }
}

// Phase 2 for one chunk (resolver wavefront).  `blocks` holds the chunk's
// block records, `aggbuf` the loaders' partial aggregates (nagg of them).
template <int G, bool PH>
__device__ void resolve_chunk(const KernelParams& P, int gidx, int k, const GroupInfo& gi,
                              float* blocks, const float* aggbuf, int nagg, int lane) {
  constexpr int REC = Cfg<G>::REC;
  const int b = gi.b, kvh = gi.kvh, T = gi.T, n_chunks = gi.n_chunks;
  const int t0 = chunk_start(P, k);
  const int nb = min(chunk_start(P, k + 1), T) - t0;
  const __amdgpu_buffer_rsrc_t rs = record_rsrc(P, gidx);
  const int rec_agg = k * 2 * P.record_floats;          // float offsets in the group's area
  const int rec_inc = rec_agg + P.record_floats;

  // the predecessor's flag, read now so that the round trip overlaps the
  // aggregate fold
  const uint64_t prev_flag = k > 0 ? ld_relaxed(P.flags + (int64_t)gidx * P.max_chunks + (k - 1)) : 0ull;
  // chunk aggregate: w0 (+) (w1 (+) w2) over the loaders' partials, or a
  // left fold over the blocks when the partials did not fit in LDS
  State<G> agg;
  if (nagg == kLoaders) {
    State<G> a1, a2;
    read_state<G>(aggbuf + 0 * REC, agg, lane);
    read_state<G>(aggbuf + 1 * REC, a1, lane);
    read_state<G>(aggbuf + 2 * REC, a2, lane);
    merge<G, false>(a1, a2);
    merge<G, false>(agg, a1);
  } else {
    State<G> t;
    state_clear<G>(agg);
    for (int i = 0; i < nb; ++i) {
      read_tile<G>(blocks + i * REC, t, lane);
      merge<G, false>(agg, t);
    }
  }

  // Softmax prefix.  Chunk 0 has an empty prefix; when chunk k-1 already
  // holds its inclusive state the prefix is that record; otherwise publish
  // the aggregate first (so that later chunks can fold past this one), look
  // back to the nearest inclusive state and fold the aggregates after it
  // forward, FW records in flight at a time.  Every path computes the same
  // left fold Agg(0) (+) ... (+) Agg(k-1), so the bits never depend on
  // timing.
  constexpr int HPL = Cfg<G>::HPL;
  constexpr int FW = 8 / HPL > 0 ? 8 / HPL : 1;
  int j;
  if (k == 0) {
    j = -1;
  } else if (flag_state(prev_flag, P.epoch) >= kInclusive) {
    j = k - 1;
  } else {
    // With few chunks of a group in flight (look_first), one pass over the
    // flags often finds the prefix complete, and the aggregate record, one
    // of the two written per chunk, is not needed by anyone; with many, the
    // later chunks need it at once to fold past this one.
    // (compiled for 8 or more heads only: the launches that pass the gate
    // are those of many groups of 8, and the extra code alone measurably
    // slowed the instances for smaller groups)
    if (G >= 8 && P.look_first) {
      // a few passes, a short sleep apart: a prefix that completes within
      // them spares this chunk its aggregate record (measured: one pass and
      // four more 0.3-0.6 % faster than one, sixteen no better, 32 slower)
      j = lookback_once(P, gidx, k, kAggregate, kInclusive, lane);
      for (int pass = 1; j == -3 && pass < kLookFirstPasses; ++pass) {
        __builtin_amdgcn_s_sleep(8);
        j = lookback_once(P, gidx, k, kAggregate, kInclusive, lane);
      }
      if (j == -3) {
        publish_state<G>(rs, rec_agg, agg, lane);
        publish(P, gidx, k, kAggregate, lane);
        j = lookback_scan(P, gidx, k, kAggregate, kInclusive, lane);
      }
    } else {
      publish_state<G>(rs, rec_agg, agg, lane);
      publish(P, gidx, k, kAggregate, lane);
      j = lookback_scan(P, gidx, k, kAggregate, kInclusive, lane);
    }
    if (j == -2) return;
  }
  stress_delay(P, gidx, k, 9);
  compiler_fence();
  State<G> pre;
  if (j >= 0) {
    fetch_state<G>(rs, j * 2 * P.record_floats + P.record_floats, pre, lane);
  } else {
    state_clear<G>(pre);
  }
  for (int i0 = j + 1; i0 < k; i0 += FW) {
    const int n = min(FW, k - i0);
    State<G> a[FW];
#pragma unroll
    for (int u = 0; u < FW; ++u)
      if (u < n) fetch_state<G>(rs, (i0 + u) * 2 * P.record_floats, a[u], lane);
#pragma unroll
    for (int u = 0; u < FW; ++u)
      if (u < n) merge<G, false>(pre, a[u]);
  }
  // this chunk's inclusive state, published before the replay: the next
  // chunks wait for it (measured: raising its flag only after the replay's
  // first blocks, to overlap the stores' completion, was 0.5 % slower)
  {
    State<G> inc = pre;
    merge<G, false>(inc, agg);
    publish_state<G>(rs, rec_inc, inc, lane);
    publish(P, gidx, k, kInclusive, lane);
    if (P.no_detector) {
      // no stability test (the detector-free baseline): later chunks need
      // only the inclusive state, and the last chunk holds the output
      if (k == n_chunks - 1) write_outputs<G>(P, b, kvh, inc, T, lane);
      return;
    }
  }

  // Replay the chunk's blocks from the prefix with the stability test.
  // Blocks go in batches of NB: the merges run in order (each needs the
  // state after the previous block) and leave per-lane partial sums of
  // |d|^2 and o(t-1).d per head; the row reductions of the whole batch then
  // run together, and |o(t)|^2 follows as |o(t-1)|^2 + 2 o(t-1).d + |d|^2.
  // The probe weights (Sec. 3.2, x = P o: 1 on the coordinates the test
  // looks at, every probe_stride-th of the head dimension, 0 elsewhere)
  // multiply the partial sums only when the probe is a subsample; this lane
  // holds coordinates 8*(lane&15) .. +7.
  constexpr int NB = 8 / HPL > 0 ? 8 / HPL : 1;
  uint32_t stable_bits = 0;
  uint32_t head_bits = 0;   // per-head mode: lane h < G, head h's stable blocks
  State<G> s = pre;   // after the replay: the state after the chunk's last block
  {
    const bool full_probe = P.probe_stride == 1;
    float pw[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      pw[e] = ((8 * (lane & 15) + e) & (P.probe_stride - 1)) == 0 ? 1.f : 0.f;
    // |x|^2 per head slot of the state before the next block
    float n_prev[HPL];
#pragma unroll
    for (int kk = 0; kk < HPL; ++kk) {
      float n0 = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) n0 = __builtin_fmaf(full_probe ? s.o[kk][e] : s.o[kk][e] * pw[e], s.o[kk][e], n0);
      n_prev[kk] = row_sum(n0);
    }
    const bool on_acc = P.scale_of_accumulator != 0;
    for (int i0 = 0; i0 < nb; i0 += NB) {
      float pdd[NB][HPL], pod[NB][HPL], pdx[NB][HPL];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
#pragma unroll
        for (int kk = 0; kk < HPL; ++kk) pdd[u][kk] = pod[u][kk] = pdx[u][kk] = 0.f;
        const int i = i0 + u;
        if (i < nb) {
          State<G> blkst;
          read_tile<G>(blocks + i * REC, blkst, lane);
          float old_o[HPL][8], old_L[HPL];
#pragma unroll
          for (int kk = 0; kk < HPL; ++kk) {
            old_L[kk] = s.L[kk];
#pragma unroll
            for (int e = 0; e < 8; ++e) old_o[kk][e] = s.o[kk][e];
          }
          float d[HPL][8];
          merge<G, true>(s, blkst, d);
#pragma unroll
          for (int kk = 0; kk < HPL; ++kk) {
            float dd = 0.f, od = 0.f, dx2 = 0.f;
            if (full_probe) {
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                dd = __builtin_fmaf(d[kk][e], d[kk][e], dd);
                od = __builtin_fmaf(old_o[kk][e], d[kk][e], od);
              }
            } else {
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                dd = __builtin_fmaf(d[kk][e] * pw[e], d[kk][e], dd);
                od = __builtin_fmaf(old_o[kk][e] * pw[e], d[kk][e], od);
              }
            }
            if (on_acc) {
              // change of the unnormalised accumulator L o, each side in its
              // own max reference (L is the mass relative to the running max)
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float dx = __fsub_rn(__fmul_rn(s.L[kk], s.o[kk][e]), __fmul_rn(old_L[kk], old_o[kk][e]));
                dx2 = __builtin_fmaf(dx * pw[e], dx, dx2);
              }
            }
            pdd[u][kk] = dd;
            pod[u][kk] = od;
            pdx[u][kk] = dx2;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < NB; ++u)
#pragma unroll
        for (int kk = 0; kk < HPL; ++kk) {
          pdd[u][kk] = row_sum(pdd[u][kk]);
          pod[u][kk] = row_sum(pod[u][kk]);
          if (on_acc) pdx[u][kk] = row_sum(pdx[u][kk]);
        }
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int i = i0 + u;
        if (i >= nb) break;
        bool ok = true;
#pragma unroll
        for (int kk = 0; kk < HPL; ++kk) {
          const float n0 = n_prev[kk], dd = pdd[u][kk], od = pod[u][kk];
          const float n1 = __fadd_rn(__fadd_rn(n0, __fmul_rn(2.f, od)), dd);   // |x(t)|^2
          n_prev[kk] = n1;
          // Eq. (2) on the probe: d_scale = |P d| (or the change of P L o);
          // d_direction = 1 - cos(P o_new, P o_old)
          const float d_scale = fast_sqrt(on_acc ? pdx[u][kk] : dd);
          const float nn = __fmul_rn(fast_sqrt(n1), fast_sqrt(n0));
          const float dot = __fadd_rn(n0, od);
          float d_dir;
          if (dot > 0.f) {
            const float num = fmaxf(__fsub_rn(__fmul_rn(n0, dd), __fmul_rn(od, od)), 0.f);
            d_dir = __fmul_rn(num, fast_rcp(__fmul_rn(nn, __fadd_rn(nn, dot))));
          } else {
            d_dir = __fsub_rn(1.f, __fmul_rn(dot, fast_rcp(nn)));
          }
          const bool st = (n0 > 0.f) && (n1 > 0.f) && (d_scale < P.tau) && (d_dir < P.phi);
          if (slot_valid<G>(lane, kk) && !st) ok = false;
          if (PH) {
            // lane h < G collects head h's verdicts: head h sits in slot
            // h / 4 of the lanes of row h % 4
            const uint64_t bal = __ballot(st);
            if (lane < G && (lane >> 2) == kk) head_bits |= (uint32_t)((bal >> (16 * (lane & 3))) & 1ull) << i;
          }
        }
        const bool all_ok = __all(ok);
        stable_bits |= (all_ok ? 1u : 0u) << i;
      }
    }
  }

  if constexpr (PH) {
    resolve_heads<G>(P, gidx, k, gi, blocks, pre, head_bits, t0, nb, lane);
    return;
  }
  // stability summary of this chunk (entering run 0)
  StabSummary sm;
  {
    int run = 0, lead = 0, fis = -1;
    bool leading = true;
    for (int i = 0; i < nb; ++i) {
      const bool st = (stable_bits >> i) & 1u;
      run = st ? run + 1 : 0;
      if (leading) {
        if (st) ++lead;
        else leading = false;
      }
      if (fis < 0 && run >= P.patience) fis = i;
    }
    sm.lead = lead;
    sm.trail = run;
    sm.len = nb;
    sm.fis = fis;
  }
  publish_word(P, gidx, k, kStabSummary, pack_summary(sm), lane);
  // A run of p stable blocks inside this chunk puts the stop here or earlier,
  // whatever the chunks before hold: the later chunks are moot from now on.
  if (sm.fis >= 0 && lane == 0) announce_stop(P, gidx, k);
  // A chunk whose first block is unstable and whose own run never reaches
  // the patience cannot hold the stop, whatever run it enters with: unless
  // it is the last chunk (which writes the untruncated result) it is done.
  if (sm.lead == 0 && sm.fis < 0 && k != n_chunks - 1) return;

  // entering stability state, then this chunk's own
  StabState x;
  stress_delay(P, gidx, k, 10);
  if (!stab_entering(P, gidx, k, x, lane)) return;
  const bool stopped_before = x.stopped != 0;
  const StabState y = stab_fold(x, sm, t0, P.patience);
  if (!stopped_before && y.stopped && sm.fis < 0 && lane == 0)  // the stop lies in this chunk
    announce_stop(P, gidx, k);
  publish_word(P, gidx, k, kStabInclusive, pack_stab(y), lane);
  if (!stopped_before && y.stopped) {
    // the stop lies in this chunk: o(t*) again from the prefix, by the same
    // merges as the replay (the same bits)
    State<G> o = pre, t;
    for (int i = 0; i < y.stop_t - t0; ++i) {
      read_tile<G>(blocks + i * REC, t, lane);
      merge<G, false>(o, t);
    }
    write_outputs<G>(P, b, kvh, o, y.stop_t, lane);
  } else if (!y.stopped && k == n_chunks - 1) {
    write_outputs<G>(P, b, kvh, s, T, lane);
  }
}

// ---- the kernel -----------------------------------------------------------------
// Persistent workgroups of four wavefronts.  Wavefronts 1..3 claim chunks
// from the work list and stream their tiles into the LDS chunk buffers in
// turn; wavefront 0 resolves earlier chunks meanwhile.  A chunk is claimed
// only once a buffer is free, and every wait targets a chunk claimed
// earlier, so the launch always makes progress.
template <int G, bool PH>
// (groups of 16 heads need the bound to keep two workgroups per CU; for
// the smaller groups the compiler's own choice was faster)
__global__ void __launch_bounds__(kThreads, G >= 16 ? 2 : 1) art_decode_kernel(const KernelParams P) {
  // the dynamic buffers must start 16-byte aligned (128-bit LDS accesses):
  // the static block below is a multiple of 16 bytes
  extern __shared__ __align__(16) float smem[];
  __shared__ __align__(16) int s_meta[kMaxSlots][8];
  // lengths of the first kLenCache sequences: a dense traversal's claims
  // need no round trip
  __shared__ __align__(16) int s_len[kLenCache];
  static_assert(sizeof(int) * (kMaxSlots * 8 + kLenCache) % 16 == 0,
                "static LDS must keep the dynamic part aligned");
  constexpr int REC = Cfg<G>::REC;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n_groups = P.batch * P.num_kv_heads;
  const int CT = P.chunk_recs_lds;
  const int nagg = P.loader_partials;
  const int slot_floats = (CT + nagg) * REC;
  const int n_slots = P.n_slots;
  // V staging buffers of the loaders after the chunk buffers (16-byte aligned)
  uint16_t* vbuf_all = reinterpret_cast<uint16_t*>(smem + ((n_slots * slot_floats + 3) & ~3));

  if (tid < kMaxSlots * 8) (&s_meta[0][0])[tid] = (tid % 8 == kMetaSeq) ? -1 : 0;
  for (int i = tid; i < min(P.batch, kLenCache); i += kThreads) s_len[i] = P.seq_lens[i];
  __syncthreads();

  if (wave == 0) {
    // ---------------- resolver ----------------
    __builtin_amdgcn_s_setprio(3);
    for (int it = 0;; ++it) {
      const int slot = it % n_slots;
      int st = kSlotFree;
      for (uint32_t spin = 0;; ++spin) {
        st = lds_ld(&s_meta[slot][kMetaState]);
        if (lds_ld(&s_meta[slot][kMetaSeq]) == it && (st == kSlotReady || st == kSlotEnd)) break;
        if (wait_expired(P, spin)) return;
        __builtin_amdgcn_s_sleep(1);
      }
      if (st == kSlotEnd) return;
      const int gidx = lds_ld(&s_meta[slot][kMetaGroup]);
      const int k = lds_ld(&s_meta[slot][kMetaChunk]);
      if (!lds_ld(&s_meta[slot][kMetaAbort])) {
        float* base = smem + slot * slot_floats;
        const GroupInfo gi = group_info_raw(P, gidx, lds_ld(&s_meta[slot][kMetaLen]),
                                            lds_ld(&s_meta[slot][kMetaListLen]));
        resolve_chunk<G, PH>(P, gidx, k, gi, base, base + CT * REC, nagg, lane);
      }
      wave_lds_sync();
      if (lane == 0) lds_st(&s_meta[slot][kMetaState], kSlotFree);
    }
  }

  // ---------------- loaders ----------------
  const int lw = wave - 1;
  // (a loader's own staging buffer: a half tile, or a quarter tile for 8 or
  // more heads; unused when V is staged in the records)
  uint16_t* vbuf = vbuf_all + lw * (G >= 8 ? 16 * kVRow : kVBufU16);
  // leader: the queue it claims from (its own first, then the others in
  // turn once its own is used up) and the queues found used up
  int qx = blockIdx.x % kQueues;
  uint64_t used_up = 0;
  constexpr uint64_t kAllUsedUp = kQueues >= 64 ? ~0ull : ((1ull << kQueues) - 1ull);

  for (int it = 0;; ++it) {
    const int slot = it % n_slots;
    if (lw == 0) {
      // leader: wait for the buffer, then claim the next chunk of the list
      bool gave_up = false;
      for (uint32_t spin = 0; lds_ld(&s_meta[slot][kMetaState]) != kSlotFree; ++spin) {
        if (wait_expired(P, spin)) {
          gave_up = true;  // hand out the end marker below
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      int gsel = -1, ksel = -1, len_sel = 0, list_sel = 0;
      while (!gave_up && used_up != kAllUsedUp) {
        const int nx = (n_groups - qx + kQueues - 1) / kQueues;  // groups in queue qx
        const int i = claim_finish(P, qx, claim_issue(P, qx, lane), lane);
        if (i >= nx * P.work_chunks) {
          used_up |= 1ull << qx;
          qx = (qx + 1) % kQueues;
          continue;
        }
        int g = qx + kQueues * (i % nx);
        const int kh = i / nx;
        // Within every full run of kQueues groups, rotate by the run's
        // index, so that each list mixes KV heads instead of holding one
        // head's groups of every sequence (whose stops can fall close
        // together and leave one list's workgroups with the late work).
        // A bijection per list: every group still belongs to one list.
        if (g / kQueues < n_groups / kQueues) g = (g / kQueues) * kQueues + (g % kQueues + g / kQueues) % kQueues;
        // the group's lengths (for a dense traversal of one of the first
        // kLenCache sequences from LDS, with no round trip); the loaders
        // check for a stop announced before the chunk with their page reads
        const int bq = g / P.num_kv_heads;
        const int L_raw = (bq < kLenCache && !P.block_list) ? lds_ld(&s_len[bq]) : P.seq_lens[bq];
        const int T_raw = raw_list_len(P, g);
        const GroupInfo gi = group_info_raw(P, g, L_raw, T_raw);
        if (gi.n_chunks == 0) {
          if (kh == 0) write_empty_wave<G>(P, gi.b, gi.kvh, lane);
          continue;
        }
        if (kh >= gi.n_chunks) continue;
        if (P.block_list && stop_word_before(ld_relaxed(P.stop_word + g), P.epoch, kh)) continue;
        gsel = g;
        ksel = kh;
        len_sel = L_raw;
        list_sel = T_raw;
        break;
      }
      // (after a give-up the buffer may still be in the resolver's hands:
      // only the end marker is handed out, its other words stay untouched)
      if (lane == 0 && !gave_up) {
        lds_st(&s_meta[slot][kMetaGroup], gsel);
        lds_st(&s_meta[slot][kMetaChunk], ksel);
        lds_st(&s_meta[slot][kMetaLen], len_sel);
        lds_st(&s_meta[slot][kMetaListLen], list_sel);
        lds_st(&s_meta[slot][kMetaDone], 0);
        lds_st(&s_meta[slot][kMetaAbort], 0);
      }
      wave_lds_sync();
      if (lane == 0) {
        lds_st(&s_meta[slot][kMetaState], gsel >= 0 ? kSlotLoading : kSlotEnd);
        lds_st(&s_meta[slot][kMetaSeq], it);
      }
    }
    // every loader: wait for this iteration's assignment
    int st = kSlotFree;
    for (uint32_t spin = 0;; ++spin) {
      st = lds_ld(&s_meta[slot][kMetaState]);
      if (lds_ld(&s_meta[slot][kMetaSeq]) == it && (st == kSlotLoading || st == kSlotEnd)) break;
      if (wait_expired(P, spin)) return;
      __builtin_amdgcn_s_sleep(1);
    }
    if (st == kSlotEnd) return;
    const int gidx = lds_ld(&s_meta[slot][kMetaGroup]);
    const int k = lds_ld(&s_meta[slot][kMetaChunk]);
    const GroupInfo gi = group_info_raw(P, gidx, lds_ld(&s_meta[slot][kMetaLen]),
                                        lds_ld(&s_meta[slot][kMetaListLen]));
    const int t0 = chunk_start(P, k);
    const int nb = min(chunk_start(P, k + 1), gi.T) - t0;
    const int tpb = P.tiles_per_block;
    float* blocks = smem + slot * slot_floats;
    bool aborted = false;
    {
      bf16x8 qa[4];
      load_q<G>(P, gi.b, gi.kvh, lane, qa);
      // This wave streams blocks lw, lw + 3, ... of the chunk, each as its
      // tpb tiles in order.  The block list entry and the pages of all its
      // tiles are fetched together once per chunk: lane 4m + n covers
      // 16-token group n of the wave's m-th tile (at most 16 tiles per wave).
      const int n_my = lw < nb ? (nb - lw + kLoaders - 1) / kLoaders * tpb : 0;
      // Bounded speculation: chunk k waits until chunk k - max_ahead of the
      // group has been through the stability test (its summary, or its
      // inclusive state without the test), unless a stop before chunk k is
      // announced meanwhile.  The waited-on chunk was claimed earlier, so
      // it makes progress without this one.
      if (P.max_ahead > 0 && k >= P.max_ahead) {
        const uint64_t* fw = P.flags + (int64_t)gidx * P.max_chunks + (k - P.max_ahead);
        const uint32_t need = P.no_detector ? kInclusive : kStabSummary;
        for (uint32_t spin = 0;; ++spin) {
          if (flag_state(ld_relaxed(fw), P.epoch) >= need) break;
          if (stop_announced_before(P, gidx, k) || wait_expired(P, spin)) {
            aborted = true;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      }
      // the stop word travels with the page reads: a chunk that lies after
      // an announced stop is given up before any tile is loaded
      const uint64_t sw0 = ld_relaxed(P.stop_word + gidx);
      int my_tok0 = 0x7fffffff, my_page = 0;
      {
        const int m = lane >> 2, n = lane & 3;
        if (m < n_my) {
          const int i = lw + kLoaders * (m / tpb), j = m % tpb;
          const int step = t0 + i;
          int blk;
          if (gi.list) {
            blk = gi.list[step];
            blk = blk < 0 ? 0 : (blk >= gi.nblk ? gi.nblk - 1 : blk);
          } else {
            blk = P.dense_order == 1 ? step : gi.nblk - 1 - step;
          }
          my_tok0 = blk * P.block_size + j * kTile;
          if (my_tok0 < gi.L) my_page = clamp_page(P, gi.b, min(my_tok0 + 16 * n, gi.L - 1));
        }
      }
      if (stop_word_before(sw0, P.epoch, k)) {
        aborted = true;
      }
      for (int m = 0; m < n_my && !aborted; ++m) {
        const int i = lw + kLoaders * (m / tpb), j = m % tpb;
        // a stop announced by an earlier chunk makes this chunk's work moot;
        // the flag read here completes while the tile's loads are in flight
        const uint64_t sw = ld_relaxed(P.stop_word + gidx);
        const int tok0 = __builtin_amdgcn_readlane(my_tok0, 4 * m);
        const int pg[4] = {__builtin_amdgcn_readlane(my_page, 4 * m), __builtin_amdgcn_readlane(my_page, 4 * m + 1),
                           __builtin_amdgcn_readlane(my_page, 4 * m + 2), __builtin_amdgcn_readlane(my_page, 4 * m + 3)};
        compute_tile<G>(P, gi.kvh, gi.L, tok0, pg, qa,
                        P.v_in_record ? reinterpret_cast<uint16_t*>(blocks + i * REC) : vbuf,
                        blocks + i * REC, j > 0);
        if (stop_word_before(sw, P.epoch, k)) {
          aborted = true;
          break;
        }
      }
    }
    wave_lds_sync();
    if (aborted) {
      if (lane == 0) lds_st(&s_meta[slot][kMetaAbort], 1);
    } else if (nagg == kLoaders) {
      // this loader's blocks folded in order: a partial aggregate
      State<G> wagg, t;
      state_clear<G>(wagg);
      for (int i = lw; i < nb; i += kLoaders) {
        read_tile<G>(blocks + i * REC, t, lane);
        merge<G, false>(wagg, t);
      }
      write_state<G>(blocks + CT * REC + lw * REC, wagg, lane);
    }
    wave_lds_sync();
    stress_delay(P, gidx, k, 13 + lw);
    if (lane == 0) {
      const int done = __hip_atomic_fetch_add(&s_meta[slot][kMetaDone], 1, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_WORKGROUP);
      if (done == kLoaders - 1) lds_st(&s_meta[slot][kMetaState], kSlotReady);
    }
  }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n_words) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words; i += stride) p[i] = 0u;
}

template <int G, bool PH>
int launch_g(const Plan& plan, const KernelParams& params, hipStream_t stream) {
  const int64_t work = (int64_t)plan.n_groups * plan.max_chunks;
  if (work <= 0) return (int)hipSuccess;
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, art_decode_kernel<G, PH>, kThreads, plan.lds_bytes);
  if (e != hipSuccess) return (int)e;
  if (per_cu < 1) per_cu = 1;
  // As many workgroups as the chip holds, but at most 32 per group (and
  // never fewer than one per CU): beyond that, a few long traversals gain
  // nothing but reads past their stops.
  const int64_t per_groups = max((int64_t)cus, (int64_t)32 * plan.n_groups);
  const int64_t grid = min(work, min((int64_t)cus * per_cu, per_groups));
  // Chunks of one group in flight at once: about the launch's chunk buffers
  // over the groups.  Up to 8 (many groups), a chunk of a group of 8 or
  // more heads looks back before it publishes its aggregate (measured: -2 %
  // on 256 groups of g = 8, +5 to +13 % with 32 or more buffers per group).
  // A function of the shape and the device only; the results are the same
  // bits either way.
  KernelParams p = params;
  p.look_first = grid * plan.slots <= (int64_t)8 * plan.n_groups ? 1 : 0;
  auto kernel = art_decode_kernel<G, PH>;
  hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(kThreads),
                     plan.lds_bytes, stream, p);
  return (int)hipGetLastError();
}

}  // namespace

int launch_decode(const Plan& plan, const KernelParams& params, hipStream_t stream) {
  switch (plan.group) {
    case 1: return params.per_head ? launch_g<1, true>(plan, params, stream) : launch_g<1, false>(plan, params, stream);
    case 2: return params.per_head ? launch_g<2, true>(plan, params, stream) : launch_g<2, false>(plan, params, stream);
    case 4: return params.per_head ? launch_g<4, true>(plan, params, stream) : launch_g<4, false>(plan, params, stream);
    case 8: return params.per_head ? launch_g<8, true>(plan, params, stream) : launch_g<8, false>(plan, params, stream);
    case 16: return params.per_head ? launch_g<16, true>(plan, params, stream) : launch_g<16, false>(plan, params, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

int launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const size_t words = bytes / 4;
  if (words == 0) return (int)hipSuccess;
  size_t blocks = (words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<uint32_t*>(ptr), words);
  return (int)hipGetLastError();
}

}  // namespace art

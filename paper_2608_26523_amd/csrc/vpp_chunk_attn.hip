// vpp_chunk_attn.hip -- chunked-prefill causal attention for MI355X (gfx950).
//
// Computes Eq. (1) of the paper (section 2.1), softmax(Q K^T * scale) V under
// the causal rule, for one chunk of query tokens at in-request positions
// prefix .. prefix+len-1 attending to the cached prefix plus the chunk itself
// (section 2.4). Several requests may share a chunk (packing, section 5.3).
//
// Kernel layout: one workgroup = 4 waves running one work slot of one query
// head: up to two query tiles of 256 (or 128) rows of one segment, the first
// with its keys ascending, the second -- its partner from the other end of the
// segment -- descending, so that the workgroups on an XCD read the same keys
// at the same time. Keys stream through LDS 64 at a time:
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: keys are the M dimension,
//     queries the N dimension, head dim the K dimension. Each lane then owns
//     one query (column lane%32) and 16 keys per 32-key block, so a row max or
//     row sum needs only one exchange with lane^32.
//   * Online softmax in fp32 with exp2 (scale folded with log2 e).
//   * O^T = V^T P^T on the same MFMA: P leaves the S^T accumulators already in
//     the B-operand layout (no shuffles); each lane reads its 8 keys of one
//     value column from the row-major V tile with two transposing 8-byte LDS
//     reads (ds_read_b64_tr_b16).
//   * Only key tiles that cross the diagonal (or the end of the key range) are
//     masked; every wave computes every key tile of its workgroup's range.
//   * Split-KV: the prefix of a segment may be cut into pieces whose fp32
//     partial results are merged by their log-sum-exp in a second pass.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <type_traits>
#include <mutex>
#include <new>
#include <vector>

#include "vpp_chunk_attn.h"

// VPP_PART: 0 = host code and the contiguous-cache kernels, 1 = the paged-cache
// kernels, 2 = the split-key-layout kernels; unset (3) = everything in one
// translation unit.
#ifndef VPP_PART
#define VPP_PART 3
#endif

namespace {

constexpr int BN = 64;         // keys per inner step
constexpr int NWAVES = 4;
// query rows per workgroup tile: 4 waves x NB blocks of 32 rows
constexpr int block_rows(int nb) { return 32 * nb * NWAVES; }
[[maybe_unused]] constexpr int BM_MAX = block_rows(2);
constexpr int NTHREADS = 64 * NWAVES;
constexpr int MAX_SPLITS = 16;
[[maybe_unused]] constexpr int STAGING_SLOTS = 4;
// cache layouts (kernel template argument KVM)
[[maybe_unused]] constexpr int KV_CONTIG = 0, KV_PAGED = 1, KV_ROPE = 2;
// split key layout: granules of the per-head and of the shared part of a K row
constexpr int NOPE_GR = 16, ROPE_GR = 8;
// Lazy rescale: the running max used for exp2 is refreshed only when a row's
// max grows past it by more than this many powers of two; O and l share the
// stale max, so the final quotient is unchanged and P stays <= 2^TAU.
constexpr float LAZY_TAU = 8.0f;
// The next tiles' global->LDS copies are spread over the first 1/LOAD_SPREAD
// of a tile's MFMA slots.
constexpr int LOAD_SPREAD = 2;
// LDS fragment prefetch distances (in fragments) of the K and V^T operands
constexpr int K_AHEAD = 3;
constexpr int V_AHEAD = 2;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// Word 3 of a raw buffer resource (untyped 32-bit data, no swizzle).
constexpr int BUFFER_RSRC_WORD3 = 0x00020000;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes): reads past the end return 0.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, int32_t bytes) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)b);
    r[1] = __builtin_amdgcn_readfirstlane((int32_t)((uint32_t)(b >> 32) & 0xffffu));  // stride 0
    r[2] = __builtin_amdgcn_readfirstlane(bytes);
    r[3] = BUFFER_RSRC_WORD3;
    return r;
}

// 16 bytes per lane from global memory (resource + per-lane byte offset)
// straight into LDS at lds_addr + 16*lane. Written as inline asm on purpose:
// the compiler then does not track these copies as pending LDS writes and
// inserts no wait for them in front of later LDS reads of other buffers; the
// kernel waits for them itself (vmcnt) before the barrier that publishes the
// buffer they fill. Nothing else in the kernel keeps a value in M0.
template <int OFF>
__device__ __forceinline__ void copy16_to_lds(const i32x4& rsrc, uint32_t lds_base, uint32_t voff) {
    // M0 = lds_base + OFF: one live SGPR for every copy of the kernel.
    // The scalar add also writes SCC: without the clobber the compiler may
    // place a copy between the two halves of a 64-bit scalar add and the high
    // half then adds the copy's carry instead of its own (an address 4 GiB off
    // whenever the low half wraps).
    asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(lds_base), "v"(voff), "s"(rsrc), "i"(OFF)
                 : "memory", "scc");
}

typedef vpp_chunk_attn_work_item_t WorkItem;
static_assert(sizeof(WorkItem) == 32, "work item layout");

}  // namespace

// Kernel argument blocks, shared by the translation units that instantiate
// the kernels (the build compiles this file once per part, in parallel).
namespace vpp_detail {

struct AttnArgs {
    const WorkItem* items;
    const u16* q;
    const u16* k;
    const u16* v;
    void* out;   // bf16 [tokens][Hq][DV]; split mode: fp32 partials [splits][tokens][Hq][DV]
    float* lse;  // fp32, h*lse_sh + row (nullable); split mode: partials [splits][Hq][tokens]
    // element strides (the host checks that they fit in 31 bits)
    int32_t q_st, q_sh, k_st, k_sh, v_st, v_sh, o_st, o_sh, lse_sh;
    int32_t num_slots;  // work slots (two work-list entries each); the grid is num_slots x num_heads
    int32_t num_entries;  // work-list entries: no entry at or past this index is read
    int32_t num_heads;
    int32_t group;     // Hq / Hkv
    int32_t tokens;    // chunk rows (partial layout)
    float scale_log2;  // softmax scale * log2(e)
    int32_t xcd_remap;
    // Paged cache (PAGED kernels only). Cache row j of segment s is row
    // j & (2^page_shift - 1) of page block_table[s * bt_st + (j >> page_shift)];
    // the work item's kv_base carries (s << 32) | its first cache row, a multiple
    // of the key tile, so no tile straddles a page (pages hold >= 64 rows).
    const int32_t* block_table;
    int64_t bt_st;
    int64_t k_sp, v_sp;  // element strides between pages
    int32_t page_shift;
    int32_t num_pages;   // page indices are clamped below it
    // Split key layout (KV_ROPE kernels only): k holds the per-head 128 dims of
    // each key, k_rope [rows][64] the 64 dims shared by all heads.
    const u16* k_rope;
    int32_t kr_st;
};

// Arguments of the merge of split partials.
struct CombineArgs {
    const float* part_o;
    const float* part_lse;
    u16* out;
    float* lse;
    int64_t o_st, o_sh, lse_sh;
    int32_t tokens, num_heads, splits;
};

hipError_t launch_attn_contig(int nb, int dqk, const AttnArgs& a, bool split, const CombineArgs& ca,
                              hipStream_t stream);
hipError_t launch_attn_paged(int nb, int dqk, const AttnArgs& a, bool split, const CombineArgs& ca,
                             hipStream_t stream);
hipError_t launch_attn_rope(int nb, const AttnArgs& a, bool split, const CombineArgs& ca, hipStream_t stream);

}  // namespace vpp_detail

namespace {

using vpp_detail::AttnArgs;
using vpp_detail::CombineArgs;

// LDS tiles: K [BN][DQK] and V [BN][DV] bf16, row-major in 16-byte granules,
// the granule index XOR-swizzled per row. The LDS serves 64 banks (256 bytes)
// per cycle:
//  * K is read by ds_read_b128, 16 lanes per cycle = 16 consecutive rows at one
//    logical granule; the 16 granules must fall on 16 different 16-byte bank
//    groups. With a multiple of 16 granules per row every row starts on the
//    same bank, so XOR with row & 15; with 8 (mod 16) granules per row
//    consecutive rows already alternate between the two 128-byte halves, so XOR
//    with (row >> 1) & 7 within each half.
//  * V is read by ds_read_b64_tr_b16, 32 lanes per cycle = 4 consecutive keys x
//    64 bytes; the four segments must fall in four different 64-byte quarters:
//    XOR with (key & 3) << 2 (16 granules per row), or with ((key >> 1) & 1) << 2
//    (8 granules per row, where odd keys already sit in the other half).
template <int KGR>
__device__ __forceinline__ int kswz(int row, int granule) {
    if constexpr (KGR % 16 == 0) return granule ^ (row & 15);
    else return granule ^ ((row >> 1) & 7);
}
template <int VGR>
__device__ __forceinline__ int vswz_bits(int key) {
    if constexpr (VGR % 16 == 0) return (key & 3) << 2;
    else return ((key >> 1) & 1) << 2;
}
template <int VGR>
__device__ __forceinline__ int vswz(int key, int granule) { return granule ^ vswz_bits<VGR>(key); }

// max of three floats in one v_max3_f32. Written as asm because the
// compiler's maxnum would first canonicalise every operand coming from an asm
// MFMA (one more VALU op per score); the scores are never NaN.
__device__ __forceinline__ float max3f(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// Plain v_max_f32: the scores are never NaN (masked ones are -inf), so the
// canonicalising maxes fmaxf would add are not needed.
__device__ __forceinline__ float max2f(float a, float b) {
    float r;
    asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ float lane_swap32_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return max2f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float lane_swap32_add(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS-only workgroup barrier: orders LDS traffic without waiting for the
// asynchronous global->LDS copies of the next stage.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// s_waitcnt with only vmcnt constrained (expcnt / lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Launch-order index -> (slot, head). With remapping on, the hardware's
// round-robin placement of consecutive workgroups on the 8 XCDs is undone so
// that each XCD runs a contiguous run of logical work (the slots of the same
// heads, which read the same K/V through that XCD's L2).
__device__ __forceinline__ void work_coords(const AttnArgs& a, int& slot, int& head) {
    const int64_t total = (int64_t)a.num_slots * a.num_heads;
    int64_t L = blockIdx.x;
    if (a.xcd_remap) {
        const int64_t per = total / 8;
        if (L < per * 8) L = (L % 8) * per + L / 8;
    }
    head = (int)(L / a.num_slots);
    slot = (int)(L % a.num_slots);
}

template <int DQK, int DV, int NB>
struct Tiles {
    static constexpr int KS = DQK / 16;          // MFMA k-steps of S^T = K Q^T
    static constexpr int DB = DV / 32;           // 32-row blocks of O^T
    static constexpr int KGR = DQK / 8;          // 16-byte granules per K row
    static constexpr int VGR = DV / 8;
    static constexpr int K_BYTES = BN * KGR * 16;
    static constexpr int V_BYTES = BN * VGR * 16;
    static constexpr int BYTES = 2 * K_BYTES + 2 * V_BYTES;  // double-buffered K and V
    static constexpr int K_LOADS = BN * KGR / 64 / NWAVES;   // 16-byte loads per lane per tile
    static constexpr int V_LOADS = BN * VGR / 64 / NWAVES;
    static constexpr int NQK = 2 * KS * NB;      // MFMAs of one S^T tile (2 key blocks x NB query blocks)
    static constexpr int NPV = 4 * DB * NB;      // MFMAs of one O^T update (4 key groups x NB query blocks)
    static_assert(KGR % 8 == 0 && VGR % 8 == 0, "swizzle needs 8 granules per row");
    static_assert(BN * KGR % (64 * NWAVES) == 0 && BN * VGR % (64 * NWAVES) == 0, "whole wave loads");
};

// S^T MFMA i of a tile: key block mb = 1 first, so that the block-0
// accumulators of the next tile are written only after the softmax has
// consumed this tile's block 0 and their registers can be reused. Within a
// key block the k-steps run in order, each K fragment feeding NB MFMAs.
template <int KS, int NB>
struct QkCoords {
    static constexpr int mb(int i) { return 1 - i / (KS * NB); }
    static constexpr int ks(int i) { return (i % (KS * NB)) / NB; }
    static constexpr int nb(int i) { return i % NB; }
};

// ---------------------------------------------------------------------------
// Static instruction schedule of one key tile.
//
// One wave (one SIMD) runs, per tile, NQK MFMAs of the next tile's S^T, NPV
// MFMAs of this tile's O^T update and the softmax of this tile in fp32 VALU
// code. A wave issues in order; VALU work issued right after an MFMA runs
// while the matrix core is busy, so the softmax is cut into small atoms
// spread over the MFMA slots. With NB query blocks of 32 rows per wave:
//   atoms 0 .. 4NB-1      4 v_max3 steps of the row max per query block
//                         (block nb = a / 4)
//   atoms 4NB .. 5NB-1    finish the row max of block nb: lane exchange, lazy
//                         rescale decision, new reference max
//   atoms 5NB .. 37NB-1   one score each: exp2, row sum, bf16 packing;
//                         element e belongs to unit u = e / 8, which holds the
//                         8 P values one O^T MFMA consumes: query block
//                         nb = u % NB, 16-key group hh = (u / NB) % 2, key
//                         block mb = u / (2 NB)
// O^T MFMA p works on key group g = p / (NB*DB) (units g*NB .. g*NB+NB-1),
// value block d = (p / NB) % DB and query block nb = p % NB, so each V^T
// fragment feeds NB MFMAs in a row; it is placed only after its group's atoms.
// All atoms finish before the last group's MFMAs start.
// ---------------------------------------------------------------------------
template <int NB>
struct Atoms {
    static constexpr int N = 37 * NB;
    static constexpr int MAXF = 4 * NB;  // first finishing atom
    static constexpr int EXP = 5 * NB;   // first exp atom
    static constexpr int weight(int k) { return k < MAXF ? 24 : (k < EXP ? 70 : 23); }  // VALU cycles
    static constexpr int unit_last(int u) { return EXP + 8 * u + 7; }
};

template <int NQK, int NPV, int DB, int NB>
struct Schedule {
    typedef Atoms<NB> A;
    // the last tile has no next S^T to overlap with: it opens with one
    // VALU-only slot for the row max, then hides each key group's atoms under
    // the previous group's MFMAs
    static constexpr int NS = NQK + NPV + (NQK == 0 ? 1 : 0);
    static constexpr int GROUP_PV = NB * DB;  // O^T MFMAs per key group
    int kind[NS] = {};      // 0: S^T MFMA, 1: O^T MFMA, 2: no MFMA
    int index[NS] = {};     // S^T: see QkCoords; O^T: see above
    int atoms_end[NS] = {}; // atoms issued after slot s: [atoms_end[s-1], atoms_end[s])
    int rescale_before = 0; // slot before which the (rare) O rescale check runs
    constexpr Schedule() {
        int done_at[A::N] = {};
        if constexpr (NQK == 0) {
            kind[0] = 2;
            for (int k = 0; k < A::EXP + 8 * NB; ++k) done_at[k] = 0;
            for (int p = 0; p < NPV; ++p) {
                kind[1 + p] = 1;
                index[1 + p] = p;
            }
            for (int g = 1; g < 4; ++g)  // key group g under group g-1's MFMAs
                for (int j = 0; j < 8 * NB; ++j)
                    done_at[A::EXP + 8 * NB * g + j] = 1 + (g - 1) * GROUP_PV + (j * GROUP_PV) / (8 * NB);
        } else {
            // slot by which each atom is done: spread by weight over the slots
            // before the last group's MFMAs
            int total = 0;
            for (int k = 0; k < A::N; ++k) total += A::weight(k);
            const int span = NS - GROUP_PV;
            int acc = 0;
            for (int k = 0; k < A::N; ++k) {
                acc += A::weight(k);
                int s = (acc * span + total - 1) / total - 1;
                done_at[k] = s < 0 ? 0 : s;
            }
            // MFMA order: an O^T MFMA as soon as its key group's atoms are done, else an S^T MFMA
            int q = 0, p = 0;
            for (int s = 0; s < NS; ++s) {
                const int grp = p / GROUP_PV;
                const bool pv_ready = p < NPV && done_at[A::EXP - 1] < s &&
                                      done_at[A::unit_last(grp * NB + NB - 1)] < s;
                if (pv_ready || q >= NQK) {
                    kind[s] = 1;
                    index[s] = p++;
                } else {
                    kind[s] = 0;
                    index[s] = q++;
                }
            }
        }
        for (int s = 0; s < NS; ++s) {
            int n = 0;
            for (int k = 0; k < A::N; ++k) n += done_at[k] <= s;
            atoms_end[s] = n;
        }
        // The (rare) O rescale is a branch; it runs right after the finishing
        // atoms. Atoms scheduled between it and the first O^T MFMA feed only code
        // after the branch, and the compiler would sink them past it into one
        // burst with no MFMA to hide under.
        rescale_before = NS;
        for (int s = NS - 1; s >= 1; --s)
            if (atoms_end[s - 1] >= A::EXP) rescale_before = s;
        for (int s = NS - 1; s >= 0; --s)
            if (kind[s] == 1 && s < rescale_before) rescale_before = s;
    }
    // MFMA slots after the last S^T MFMA of the step
    constexpr int qk_tail() const {
        int last = -1;
        for (int s = 0; s < NS; ++s)
            if (kind[s] == 0) last = s;
        return NS - 1 - last;
    }
    // every O^T MFMA comes after the atoms it depends on; atoms run in order
    constexpr bool valid() const {
        for (int s = 0; s < NS; ++s) {
            if (s > 0 && atoms_end[s] < atoms_end[s - 1]) return false;
            if (kind[s] != 1) continue;
            const int grp = index[s] / GROUP_PV;
            const int before = s == 0 ? 0 : atoms_end[s - 1];
            if (before < A::unit_last(grp * NB + NB - 1) + 1) return false;
        }
        return atoms_end[NS - 1] == A::N;
    }
};

// The S^T MFMAs are inline asm so that each operand stays in the register
// file it belongs to for the whole loop: S in VGPRs (the softmax reads and
// writes it in place) and Q in AGPRs (only MFMAs read it). The compiler cannot
// see the latency of these instructions, so the schedule keeps the distance
// itself: an S^T tile is read by VALU code only in the next tile's step (after
// a barrier), and every step ends with at least four O^T MFMAs after its last
// S^T MFMA (checked in the kernel), each occupying the matrix core for longer
// than an S^T result takes to reach its registers. The O^T MFMAs use the
// builtin, so the compiler tracks their operand hazards (P packed by VALU code
// just before) and keeps O in AGPRs; the asm that rescales O in place runs only
// after an explicit drain.
#define MFMA_32x32x16_INIT(acc, a, b) \
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "a"(b))
#define MFMA_32x32x16_ACC(acc, a, b) \
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "a"(b))

__device__ __forceinline__ void mfma_drain() {
    // longer than the longest MFMA result latency: 3 x 16 wait states
    asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
}

// Load the KS B-operand fragments of one query row (16 bytes each, 32 bytes
// apart) straight into AGPRs, where only MFMAs read them. Loading through
// VGPRs would leave a VGPR copy of Q alive across the whole loop.
template <int KS>
__device__ __forceinline__ void load_q_agpr(bf16x8 (&qf)[KS], const void* p) {
    static_assert(KS == 4 || KS == 8 || KS == 12, "head dims 64, 128, 192");
    if constexpr (KS == 4) {
        asm volatile(
            "global_load_dwordx4 %0, %4, off\n\t"
            "global_load_dwordx4 %1, %4, off offset:32\n\t"
            "global_load_dwordx4 %2, %4, off offset:64\n\t"
            "global_load_dwordx4 %3, %4, off offset:96"
            : "=a"(qf[0]), "=a"(qf[1]), "=a"(qf[2]), "=a"(qf[3])
            : "v"(p) : "memory");
    } else if constexpr (KS == 8) {
        asm volatile(
            "global_load_dwordx4 %0, %8, off\n\t"
            "global_load_dwordx4 %1, %8, off offset:32\n\t"
            "global_load_dwordx4 %2, %8, off offset:64\n\t"
            "global_load_dwordx4 %3, %8, off offset:96\n\t"
            "global_load_dwordx4 %4, %8, off offset:128\n\t"
            "global_load_dwordx4 %5, %8, off offset:160\n\t"
            "global_load_dwordx4 %6, %8, off offset:192\n\t"
            "global_load_dwordx4 %7, %8, off offset:224"
            : "=a"(qf[0]), "=a"(qf[1]), "=a"(qf[2]), "=a"(qf[3]), "=a"(qf[4]), "=a"(qf[5]),
              "=a"(qf[6]), "=a"(qf[7])
            : "v"(p) : "memory");
    } else {
        asm volatile(
            "global_load_dwordx4 %0, %12, off\n\t"
            "global_load_dwordx4 %1, %12, off offset:32\n\t"
            "global_load_dwordx4 %2, %12, off offset:64\n\t"
            "global_load_dwordx4 %3, %12, off offset:96\n\t"
            "global_load_dwordx4 %4, %12, off offset:128\n\t"
            "global_load_dwordx4 %5, %12, off offset:160\n\t"
            "global_load_dwordx4 %6, %12, off offset:192\n\t"
            "global_load_dwordx4 %7, %12, off offset:224\n\t"
            "global_load_dwordx4 %8, %12, off offset:256\n\t"
            "global_load_dwordx4 %9, %12, off offset:288\n\t"
            "global_load_dwordx4 %10, %12, off offset:320\n\t"
            "global_load_dwordx4 %11, %12, off offset:352"
            : "=a"(qf[0]), "=a"(qf[1]), "=a"(qf[2]), "=a"(qf[3]), "=a"(qf[4]), "=a"(qf[5]),
              "=a"(qf[6]), "=a"(qf[7]), "=a"(qf[8]), "=a"(qf[9]), "=a"(qf[10]), "=a"(qf[11])
            : "v"(p) : "memory");
    }
}

// o *= alpha for one 16-AGPR accumulator tile, in place, through a single
// temporary VGPR (the accumulators never get a VGPR home).
__device__ __forceinline__ void scale_agpr_tile(f32x16& o, float alpha) {
    float e0 = o[0], e1 = o[1], e2 = o[2], e3 = o[3], e4 = o[4], e5 = o[5], e6 = o[6], e7 = o[7];
    float e8 = o[8], e9 = o[9], e10 = o[10], e11 = o[11], e12 = o[12], e13 = o[13], e14 = o[14], e15 = o[15];
    float tmp;
#define SCALE_ONE(n) "v_accvgpr_read_b32 %16, %" #n "\n\ts_nop 1\n\tv_mul_f32 %16, %16, %17\n\ts_nop 1\n\tv_accvgpr_write_b32 %" #n ", %16\n\t"
    asm volatile(SCALE_ONE(0) SCALE_ONE(1) SCALE_ONE(2) SCALE_ONE(3) SCALE_ONE(4) SCALE_ONE(5) SCALE_ONE(6)
                 SCALE_ONE(7) SCALE_ONE(8) SCALE_ONE(9) SCALE_ONE(10) SCALE_ONE(11) SCALE_ONE(12) SCALE_ONE(13)
                 SCALE_ONE(14) SCALE_ONE(15) "s_nop 1"
                 : "+a"(e0), "+a"(e1), "+a"(e2), "+a"(e3), "+a"(e4), "+a"(e5), "+a"(e6), "+a"(e7), "+a"(e8),
                   "+a"(e9), "+a"(e10), "+a"(e11), "+a"(e12), "+a"(e13), "+a"(e14), "+a"(e15), "=&v"(tmp)
                 : "v"(alpha));
#undef SCALE_ONE
    o[0] = e0; o[1] = e1; o[2] = e2; o[3] = e3; o[4] = e4; o[5] = e5; o[6] = e6; o[7] = e7;
    o[8] = e8; o[9] = e9; o[10] = e10; o[11] = e11; o[12] = e12; o[13] = e13; o[14] = e14; o[15] = e15;
}

template <int N, typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>()), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl<N>(f, std::make_integer_sequence<int, N>());
}
// f(A0), f(A0 + 1), ..., f(A1 - 1)
template <int A0, typename F, int... I>
__device__ __forceinline__ void static_range_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, A0 + I>()), ...);
}
template <int A0, int A1, typename F>
__device__ __forceinline__ void static_range(F&& f) {
    static_range_impl<A0>(f, std::make_integer_sequence<int, A1 - A0>());
}

// NB = 2: 64 query rows per wave, one workgroup (4 waves) per CU. NB = 1: 32
// rows per wave and half the registers, so two workgroups share a CU and each
// SIMD interleaves two waves' instruction streams.
// KVM: the cache layout. KV_CONTIG: K [rows][Hkv][dqk] and V [rows][Hkv][dv];
// KV_PAGED: the same rows in pages reached through a block table; KV_ROPE
// (dqk = 192 only): K split into a per-head part k_nope [rows][Hkv][128] and a
// part shared by all heads k_rope [rows][64], the key layout of the MLA models.
template <int DQK, int DV, int NB, bool SPLIT, int KVM>
__global__ __attribute__((amdgpu_flat_work_group_size(NTHREADS, NTHREADS), amdgpu_waves_per_eu(3 - NB, 3 - NB)))
void attn_fwd_kernel(AttnArgs a) {
    constexpr bool PAGED = KVM == KV_PAGED;
    constexpr bool ROPE = KVM == KV_ROPE;
    static_assert(!ROPE || DQK == 192, "the split key layout is 128 + 64 dims");
    typedef Tiles<DQK, DV, NB> T;
    typedef Atoms<NB> A;
    constexpr int KS = T::KS;
    constexpr int DB = T::DB;
    constexpr int WROWS = 32 * NB;  // query rows per wave
    typedef Schedule<T::NQK, T::NPV, DB, NB> SchedFull;
    typedef Schedule<0, T::NPV, DB, NB> SchedLast;
    static_assert(SchedFull().valid() && SchedLast().valid(), "tile schedule breaks a dependency");
    static_assert(SchedFull().qk_tail() >= 4, "the next step's softmax could read S^T before it lands");

    __shared__ __attribute__((aligned(1024))) char smem[T::BYTES];
    char* const kbuf0 = smem;
    char* const vbuf0 = smem + 2 * T::K_BYTES;

    int slot, h;
    work_coords(a, slot, h);
    // A slot holds up to two tiles: the first runs its key range ascending, the
    // second (if any) descending; an empty second entry has no rows.
#pragma nounroll
    for (int sub = 0; sub < 2; ++sub) {
        const int item_id = 2 * slot + sub;
        if (item_id >= a.num_entries) break;
        // the work item is uniform: keep it in SGPRs (so buffer resources built
        // from it are scalar too)
        WorkItem it = a.items[item_id];
        it.row0 = __builtin_amdgcn_readfirstlane(it.row0);
        it.nrows = __builtin_amdgcn_readfirstlane(it.nrows);
        it.pos0 = __builtin_amdgcn_readfirstlane(it.pos0);
        it.key_begin = __builtin_amdgcn_readfirstlane(it.key_begin);
        it.key_end = __builtin_amdgcn_readfirstlane(it.key_end);
        it.split = __builtin_amdgcn_readfirstlane(it.split);
        it.kv_base = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(it.kv_base >> 32)) << 32) |
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)it.kv_base));
        if (it.nrows == 0) break;
        // every wave is done with the LDS tiles of the slot's previous tile before
        // this tile's first copies overwrite them
        lds_barrier();
        const int hk = h / a.group;
        const int tid = threadIdx.x;
        const int lane = tid & 63;
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS bases stay scalar
        const int lr = lane & 31;
        const int lg = lane >> 5;

        const int kb = it.key_begin, ke = it.key_end;
        // contiguous cache: the request's row 0 of head hk; paged: page 0's row 0
        const int64_t cache_row0 = PAGED ? 0 : it.kv_base;
        const u16* kbase = a.k + cache_row0 * a.k_st + (int64_t)hk * a.k_sh;
        const u16* vbase = a.v + cache_row0 * a.v_st + (int64_t)hk * a.v_sh;
        const int ntiles = (ke - kb + BN - 1) / BN;
        // key tiles sit at kb + m*BN (m = 0 .. ntiles-1) in both directions; visit j
        // of the tile loop reads the tile at kt_first + j*dkt
        const bool rev = sub != 0;
        const int dkt = rev ? -BN : BN;
        const int kt_first = rev ? kb + (ntiles - 1) * BN : kb;
        // paged cache: this segment's block-table row and the cache row of key 0
        const int32_t* bt_row = PAGED ? a.block_table + (int64_t)(int32_t)(it.kv_base >> 32) * a.bt_st : nullptr;
        const int kv_off = PAGED ? (int)(uint32_t)it.kv_base : 0;
        const int pmask = PAGED ? (1 << a.page_shift) - 1 : 0;
        const int last_row = kv_off + ke - 1;  // page reads past the key range are clamped here
        auto clamp_page = [&](int pg) { return (int)min((uint32_t)pg, (uint32_t)(a.num_pages - 1)); };
        auto page_of = [&](int row) {  // synchronous lookup (prologue)
            return clamp_page(__builtin_amdgcn_readfirstlane(bt_row[min(row, last_row) >> a.page_shift]));
        };
        // first element of the tile of keys starting at kt
        auto tile_src = [&](const u16* base, int64_t page_st, int64_t row_st, int kt) -> const u16* {
            if constexpr (PAGED) {
                const int row = kv_off + kt;
                return base + (int64_t)page_of(row) * page_st + (int64_t)(row & pmask) * row_st;
            } else {
                return base + (int64_t)kt * row_st;
            }
        };

        // This lane's NB query rows (one per 32-column block of S^T), as B
        // operands in AGPRs. Rows past the tile re-read its last row (their results
        // are never stored), so every load stays inside q.
        bf16x8 qf[NB][KS];
        int qlim[NB];   // last key position the row may see, minus lg*4 (see masking)
        bool qvalid[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int rloc = wave * WROWS + nb * 32 + lr;
            qvalid[nb] = rloc < it.nrows;
            qlim[nb] = min(it.pos0 + rloc, ke - 1) - lg * 4;
            const u16* qp = a.q + (int64_t)(it.row0 + min(rloc, it.nrows - 1)) * a.q_st + (int64_t)h * a.q_sh + lg * 8;
            load_q_agpr<KS>(qf[nb], qp);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        const int wave_first = it.pos0 + wave * WROWS;

        // Global->LDS copy of one tile through a buffer resource whose base is the
        // tile's first key row and whose size ends at the last key of the range:
        // rows past the range read as zeros (buffer range check), so the last tile
        // needs no special case. Per-lane byte offsets are fixed for the kernel.
        // Split key layout: the K tile is two LDS regions, the per-head part
        // [BN][NOPE_GR] granules then the shared part [BN][ROPE_GR], each filled by
        // its own copies (a copy instruction has one source) and swizzled for its
        // own row width; the first NOPE_LOADS copies read k_nope, the rest k_rope.
        constexpr int NOPE_LOADS = BN * NOPE_GR / NTHREADS;
        constexpr int NOPE_BYTES = BN * NOPE_GR * 16;
        uint32_t k_src[T::K_LOADS], v_src[T::V_LOADS];
#pragma unroll
        for (int t = 0; t < T::K_LOADS; ++t) {
            if constexpr (ROPE) {
                if (t < NOPE_LOADS) {
                    const int slot = t * NTHREADS + tid;
                    const int row = slot / NOPE_GR, gs = slot % NOPE_GR;
                    k_src[t] = (uint32_t)(row * (int)a.k_st + kswz<NOPE_GR>(row, gs) * 8) * 2u;
                } else {
                    const int slot = (t - NOPE_LOADS) * NTHREADS + tid;
                    const int row = slot / ROPE_GR, gs = slot % ROPE_GR;
                    k_src[t] = (uint32_t)(row * (int)a.kr_st + kswz<ROPE_GR>(row, gs) * 8) * 2u;
                }
            } else {
                const int slot = t * NTHREADS + tid;
                const int row = slot / T::KGR, gs = slot % T::KGR;
                k_src[t] = (uint32_t)(row * (int)a.k_st + kswz<T::KGR>(row, gs) * 8) * 2u;
            }
        }
#pragma unroll
        for (int t = 0; t < T::V_LOADS; ++t) {
            const int slot = t * NTHREADS + tid;
            const int row = slot / T::VGR, gs = slot % T::VGR;
            v_src[t] = (uint32_t)(row * (int)a.v_st + vswz<T::VGR>(row, gs) * 8) * 2u;
        }
        // resources over the rows [kt, min(kt + BN, ke)) (none when kt >= ke); the host
        // keeps row strides below 2^31 / (2 BN) elements, so a tile's byte count fits
        auto tile_bytes = [&](int kt, int32_t row_st) {
            return (int32_t)((uint32_t)max(0, min(BN, ke - kt)) * (uint32_t)row_st * 2u);
        };
        auto k_rsrc = [&](int kt) { return make_rsrc(tile_src(kbase, a.k_sp, a.k_st, kt), tile_bytes(kt, a.k_st)); };
        // the shared key part of the same rows (split layout; one row per key, no head)
        const u16* rbase = ROPE ? a.k_rope + cache_row0 * a.kr_st : nullptr;
        auto kr_rsrc = [&](int kt) { return make_rsrc(rbase + (int64_t)kt * a.kr_st, tile_bytes(kt, a.kr_st)); };
        auto v_rsrc = [&](int kt) { return make_rsrc(tile_src(vbase, a.v_sp, a.v_st, kt), tile_bytes(kt, a.v_st)); };
        const uint32_t lds_wave = (uint32_t)(uintptr_t)(lds_void_t*)smem + (uint32_t)wave * 1024u;
        // copy t of the K (V) tile into buffer B: LDS offset from this wave's base
        auto load_k = [&](const i32x4& r, const i32x4& rr, auto B, auto TT) {
            constexpr int t = decltype(TT)::value;
            if constexpr (ROPE && t >= NOPE_LOADS) {
                constexpr int off = decltype(B)::value * T::K_BYTES + NOPE_BYTES + (t - NOPE_LOADS) * NWAVES * 1024;
                copy16_to_lds<off>(rr, lds_wave, k_src[t]);
            } else {
                constexpr int off = decltype(B)::value * T::K_BYTES + t * NWAVES * 1024;
                copy16_to_lds<off>(r, lds_wave, k_src[t]);
            }
        };
        auto load_v = [&](const i32x4& r, auto B, auto TT) {
            constexpr int off = 2 * T::K_BYTES + decltype(B)::value * T::V_BYTES + decltype(TT)::value * NWAVES * 1024;
            copy16_to_lds<off>(r, lds_wave, v_src[decltype(TT)::value]);
        };
        auto issue_k = [&](auto B, int kt) {
            const i32x4 r = k_rsrc(kt);
            const i32x4 rr = ROPE ? kr_rsrc(kt) : r;
            static_for<T::K_LOADS>([&](auto TT) { load_k(r, rr, B, TT); });
        };
        auto issue_v = [&](auto B, int kt) {
            const i32x4 r = v_rsrc(kt);
            static_for<T::V_LOADS>([&](auto TT) { load_v(r, B, TT); });
        };
        if (ntiles > 0) {
            issue_k(std::integral_constant<int, 0>(), kt_first);
            issue_v(std::integral_constant<int, 0>(), kt_first);
            if (ntiles > 1) issue_k(std::integral_constant<int, 1>(), kt_first + dkt);
        }

        // Per-lane LDS byte offsets; the rest of each address is an immediate.
        // K (A operand of S^T): row mb*32+lr, logical granule ks*2+lg; row & 15 and
        // (row >> 1) & 7 depend only on lr. The swizzle touches the low 4 (or 3)
        // bits of the granule index, so K_OFFS offsets cover every ks and the
        // higher granule bits are an immediate.
        // (split key layout: K_OFFS offsets for the per-head region, KR_OFFS for the
        // shared one)
        constexpr int K_OFFS = ROPE ? NOPE_GR / 2 : ((T::KGR % 16 == 0) ? 8 : 4);
        constexpr int KR_OFFS = ROPE ? ROPE_GR / 2 : 1;
        int k_off[K_OFFS], kr_off[KR_OFFS];
#pragma unroll
        for (int r = 0; r < K_OFFS; ++r) {
            if constexpr (ROPE) k_off[r] = lr * (NOPE_GR * 16) + kswz<NOPE_GR>(lr, r * 2 + lg) * 16;
            else k_off[r] = lr * (T::KGR * 16) + kswz<T::KGR>(lr, r * 2 + lg) * 16;
        }
#pragma unroll
        for (int r = 0; r < KR_OFFS; ++r) kr_off[r] = ROPE ? lr * (ROPE_GR * 16) + kswz<ROPE_GR>(lr, r * 2 + lg) * 16 : 0;
        // V^T (A operand of O^T) through ds_read_b64_tr_b16: 16-lane group q reads
        // keys 4*(q>>1) + (j>>2) and value columns 16*(q&1) + 4*(j&3) .. +3, i.e.
        // granule 4*d + (tr_col >> 3) of value block d; key & 3 = tr_key & 3.
        const int tq = lane >> 4, tj = lane & 15;
        const int tr_key = 4 * (tq >> 1) + (tj >> 2);
        const int tr_col = 16 * (tq & 1) + 4 * (tj & 3);
        int v_off[DB];
#pragma unroll
        for (int d = 0; d < DB; ++d)
            v_off[d] = tr_key * (T::VGR * 16) + vswz<T::VGR>(tr_key, d * 4 + (tr_col >> 3)) * 16 + (tr_col & 7) * 2;

        float m_run[NB];   // max used by exp2 (log2 units), refreshed lazily
        float l_part[NB];  // this lane's share of the softmax denominator
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            m_run[nb] = -INFINITY;
            l_part[nb] = 0.f;
        }
        f32x16 o[DB][NB];
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int i = 0; i < 16; ++i) o[d][nb][i] = 0.f;

        auto load_kfrag = [&](const char* kt_buf, int ks, int mb) -> bf16x8 {
            if constexpr (ROPE) {
                const char* addr = ks < NOPE_GR / 2
                                       ? kt_buf + mb * 32 * NOPE_GR * 16 + k_off[ks]
                                       : kt_buf + NOPE_BYTES + mb * 32 * ROPE_GR * 16 + kr_off[ks - NOPE_GR / 2];
                return __builtin_bit_cast(bf16x8, *(const u32x4*)addr);
            } else {
                const u32x4 raw = *(const u32x4*)(kt_buf + mb * 32 * T::KGR * 16 + (ks / K_OFFS) * (K_OFFS * 32) +
                                                  k_off[ks % K_OFFS]);
                return __builtin_bit_cast(bf16x8, raw);
            }
        };
        auto load_vfrag = [&](const char* vt, int mb, int hh, int d) -> bf16x8 {
            bf16x8 af;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const char* addr = vt + (mb * 32 + hh * 16 + half * 8) * T::VGR * 16 + v_off[d];
                const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(addr));
                const bf16x4 rb = __builtin_bit_cast(bf16x4, r);
#pragma unroll
                for (int j = 0; j < 4; ++j) af[half * 4 + j] = rb[j];
            }
            return af;
        };

        // S^T = K Q^T for a whole tile (prologue only: no softmax to overlap with)
        auto qk_all = [&](const char* kt_buf, f32x16 (&s)[2][NB]) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const bf16x8 af = load_kfrag(kt_buf, ks, mb);
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const bf16x8 bq = qf[nb][ks];
                        if (ks == 0) MFMA_32x32x16_INIT(s[mb][nb], af, bq);
                        else MFMA_32x32x16_ACC(s[mb][nb], af, bq);
                    }
                }
        };

        // Running sources of the copies a step issues (K of visit t+2, V of visit
        // t+1): scalar pointer, first key and visits left, advanced by one tile per
        // step. Past the last visit a copy gets an empty resource; its pointer may
        // then run outside the tensor, but an empty resource never reads it.
        const uint32_t k_row_bytes = (uint32_t)a.k_st * 2u, v_row_bytes = (uint32_t)a.v_st * 2u;
        // V of visit t+1 is one visit behind K of visit t+2: its first key is
        // kt_k - dkt and it has one visit more left
        uint64_t k_next = PAGED ? 0 : (uint64_t)(uintptr_t)kbase + (uint64_t)((int64_t)(kt_first + 2 * dkt) * k_row_bytes);
        uint64_t v_next = PAGED ? 0 : (uint64_t)(uintptr_t)vbase + (uint64_t)((int64_t)(kt_first + dkt) * v_row_bytes);
        int kt_k = kt_first + 2 * dkt;
        int k_left = ntiles - 2;
        // split key layout: the shared part's running source (same rows as K)
        const uint32_t kr_row_bytes = ROPE ? (uint32_t)a.kr_st * 2u : 0u;
        uint64_t kr_next = ROPE ? (uint64_t)(uintptr_t)rbase + (uint64_t)((int64_t)(kt_first + 2 * dkt) * kr_row_bytes) : 0;
        // one tile of rows in bytes (below 2^31), signed by the direction
        auto tile_step = [&](uint32_t row_bytes) { return (uint64_t)(int64_t)(rev ? -(int32_t)(BN * row_bytes) : (int32_t)(BN * row_bytes)); };
        // paged cache: the page of the K tile a step copies is read one step ahead
        // (raw, clamped at its use), and V(t+1) shares K(t+1)'s page; table reads
        // are clamped to the rows of the key range
        auto clamp_row = [&](int row) { return min(max(row, kv_off + kb), last_row); };
        int pg_pending = 0, pg_prev = 0;
        if constexpr (PAGED) {
            if (ntiles > 0) {
                pg_prev = page_of(clamp_row(kv_off + kt_first + dkt));
                pg_pending = bt_row[clamp_row(kv_off + kt_first + 2 * dkt) >> a.page_shift];
            }
        }

        // One key tile: mask S(t) if needed, then the scheduled mix of S(t+1)
        // MFMAs, the softmax of S(t) and the O^T += V^T P^T MFMAs of tile t.
        auto step = [&](auto P, auto HAS_NEXT, int t, f32x16 (&s_cur)[2][NB], f32x16 (&s_nxt)[2][NB]) {
            constexpr int par = decltype(P)::value;
            constexpr bool has_next = decltype(HAS_NEXT)::value;
            const char* kt_nxt = kbuf0 + (1 - par) * T::K_BYTES;
            const char* vt_cur = vbuf0 + par * T::V_BYTES;
            const int kt = kt_first + t * dkt;
            wait_vmcnt<0>();
            lds_barrier();  // K(t+1), V(t) are in LDS; every wave is done with K(t) and V(t-1)
            // the next tiles' copies (K(t+2) into the K buffer just freed, V(t+1)
            // into the V buffer just freed) are spread over the first slots. Past
            // the last tile the resources are empty: the copies then only write
            // zeros into buffers that no later step reads, and the step needs no
            // branch around them.
            if constexpr (PAGED) {
                // the page read during the previous step is complete after the
                // barrier; the empty asm pins its use here, before any LDS read of
                // this step is in flight
                int pg_k = clamp_page(__builtin_amdgcn_readfirstlane(pg_pending));
                asm volatile("" : "+s"(pg_k) : : "memory");
                const int row_k = kv_off + kt_k, row_v = row_k - dkt;
                k_next = (uint64_t)(uintptr_t)(kbase + (int64_t)pg_k * a.k_sp + (int64_t)(row_k & pmask) * a.k_st);
                v_next = (uint64_t)(uintptr_t)(vbase + (int64_t)pg_prev * a.v_sp + (int64_t)(row_v & pmask) * a.v_st);
                pg_prev = pg_k;
                pg_pending = bt_row[clamp_row(row_k + dkt) >> a.page_shift];
            }
            // rows of the copied tile (a tile is partial only at the end of the
            // range), times the row bytes (below 2^31); none past the last visit
            const uint32_t k_n = k_left > 0 ? (uint32_t)min(BN, ke - kt_k) : 0u;
            const uint32_t v_n = k_left >= 0 ? (uint32_t)min(BN, ke - (kt_k - dkt)) : 0u;
            const i32x4 rk = make_rsrc((const void*)k_next, (int32_t)(k_n * k_row_bytes));
            const i32x4 rv = make_rsrc((const void*)v_next, (int32_t)(v_n * v_row_bytes));
            i32x4 rkr = rk;
            if constexpr (ROPE) {
                rkr = make_rsrc((const void*)kr_next, (int32_t)(k_n * kr_row_bytes));
                kr_next += tile_step(kr_row_bytes);
            }
            if constexpr (!PAGED) {
                k_next += tile_step(k_row_bytes);
                v_next += tile_step(v_row_bytes);
            }
            kt_k += dkt;
            --k_left;

            // causal / range mask on the tiles that cross a row's last visible key:
            // key kt + c (c = mb*32 + (i>>2)*8 + lg*4 + (i&3)) is hidden when
            // c > qlim - kt, with qlim = min(row position, ke - 1) - lg*4
            if ((kt + BN - 1 > wave_first) || (kt + BN > ke)) {
                const float ninf = -INFINITY;
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int lim = qlim[nb] - kt;
#pragma unroll
                    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            // compare and select through VCC, one element at a time (no
                            // batch of 64-bit lane masks in scalar registers)
                            float x = s_cur[mb][nb][i];
                            asm("v_cmp_gt_i32 vcc, %2, %1\n\tv_cndmask_b32 %0, %0, %3, vcc"
                                : "+v"(x)
                                : "v"(lim), "i"(mb * 32 + (i >> 2) * 8 + (i & 3)), "v"(ninf)
                                : "vcc");
                            s_cur[mb][nb][i] = x;
                        }
                }
            }

            float alpha[NB], m_use[NB], mx[NB][4], lsum[NB][2];  // mx: one partial max per max atom
            bool refresh[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                alpha[nb] = 1.f;
                m_use[nb] = 0.f;
                lsum[nb][0] = lsum[nb][1] = 0.f;
                refresh[nb] = false;
            }
            float pprev = 0.f;
            bf16x8 pb[NB][2][2];         // [nb][mb][hh]
            bf16x8 kf[K_AHEAD + 1];      // K fragments in issue order, K_AHEAD in flight
            bf16x8 vf[V_AHEAD + 1];      // V^T fragments in issue order, V_AHEAD in flight

            auto atom = [&](auto K) {
                constexpr int k = decltype(K)::value;
                if constexpr (k < A::MAXF) {
                    // max of 8 of the 32 scores of query block nb, as a depth-2 tree:
                    // the four atoms of a row are independent of each other
                    constexpr int nb = k >> 2, q = k & 3;
                    auto sc = [&](int j) -> float {
                        const int v = q * 8 + j;  // score index in [mb*16 + i]
                        return s_cur[v >> 4][nb][v & 15];
                    };
                    const float t0 = max3f(sc(0), sc(1), sc(2));
                    const float t1 = max3f(sc(3), sc(4), sc(5));
                    const float t2 = max2f(sc(6), sc(7));
                    mx[nb][q] = max3f(t0, t1, t2);
                } else if constexpr (k < A::EXP) {
                    constexpr int nb = k - A::MAXF;
                    const float m =
                        lane_swap32_max(max3f(mx[nb][0], mx[nb][1], max2f(mx[nb][2], mx[nb][3]))) * a.scale_log2;
                    // per-lane decision: the exps of this row wait only for VALU work;
                    // the wave-wide vote happens once, at the rescale check
                    refresh[nb] = m > m_run[nb] + LAZY_TAU;
                    const float m_new = refresh[nb] ? m : m_run[nb];
                    // a row that has seen no visible key yet (m_new = -inf) has nothing to rescale
                    alpha[nb] = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run[nb] - m_new);
                    m_run[nb] = m_new;
                    m_use[nb] = (m_new == -INFINITY) ? 0.f : m_new;
                    l_part[nb] *= alpha[nb];
                } else {
                    constexpr int e = k - A::EXP;
                    constexpr int u = e >> 3, j = e & 7;
                    constexpr int mb = u / (2 * NB), hh = (u / NB) & 1, nb = u % NB;
                    const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s_cur[mb][nb][hh * 8 + j], a.scale_log2, -m_use[nb]));
                    lsum[nb][j & 1] += pv;
                    if constexpr ((j & 1) == 0) {
                        pprev = pv;
                    } else {
                        pb[nb][mb][hh][j - 1] = (__bf16)pprev;
                        pb[nb][mb][hh][j] = (__bf16)pv;
                    }
                }
            };

            auto run = [&](auto tag) {
                typedef typename decltype(tag)::type Sch;
                constexpr Sch sch{};
                constexpr int NS = Sch::NS;
                typedef QkCoords<KS, NB> C;
                // fragments needed first: V_AHEAD V^T fragments, and K_AHEAD K fragments of the next tile
                static_for<V_AHEAD>([&](auto I) {
                    constexpr int f = I;
                    vf[f] = load_vfrag(vt_cur, (f / DB) >> 1, (f / DB) & 1, f % DB);
                });
                if constexpr (has_next)
                    static_for<K_AHEAD>([&](auto I) {
                        constexpr int f = I;
                        kf[f] = load_kfrag(kt_nxt, C::ks(NB * f), C::mb(NB * f));
                    });
                static_for<NS>([&](auto SL) {
                    constexpr int s = SL;
                    constexpr int kind = sch.kind[s];
                    constexpr int idx = sch.index[s];
                    if constexpr (s == sch.rescale_before) {
                        bool any = false;
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb) any = any || refresh[nb];
                        if (__builtin_amdgcn_ballot_w64(any) != 0) {
                            // rare: rescale the AGPR accumulators 16 at a time, so the
                            // branch needs only a few temporary VGPRs (alpha = 1 in the
                            // lanes whose reference did not move)
                            mfma_drain();
                            static_for<NB * DB>([&](auto J) {
                                constexpr int nb = J / DB, d = J % DB;
                                scale_agpr_tile(o[d][nb], alpha[nb]);
                                __builtin_amdgcn_sched_barrier(0);
                            });
                        }
                    }
                    if constexpr (has_next) {
                        constexpr int NL = T::K_LOADS + T::V_LOADS;
                        constexpr int LSTRIDE = (NS / LOAD_SPREAD) / NL > 0 ? (NS / LOAD_SPREAD) / NL : 1;
                        if constexpr (s % LSTRIDE == 0 && s / LSTRIDE < NL) {
                            constexpr int j = s / LSTRIDE;
                            if constexpr (j < T::V_LOADS) {
                                load_v(rv, std::integral_constant<int, 1 - par>(), std::integral_constant<int, j>());
                            } else {
                                load_k(rk, rkr, std::integral_constant<int, par>(),
                                       std::integral_constant<int, j - T::V_LOADS>());
                            }
                        }
                    }
                    if constexpr (kind == 2) {
                        // VALU-only slot
                    } else if constexpr (kind == 0) {
                        constexpr int ks = C::ks(idx), mb = C::mb(idx), nb = C::nb(idx);
                        constexpr int frag = idx / NB;  // (mb, ks) in issue order
                        // prefetch K_AHEAD fragments ahead with this fragment's first MFMA
                        if constexpr (nb == 0 && frag + K_AHEAD < 2 * KS)
                            kf[(frag + K_AHEAD) % (K_AHEAD + 1)] =
                                load_kfrag(kt_nxt, C::ks(NB * (frag + K_AHEAD)), C::mb(NB * (frag + K_AHEAD)));
                        const bf16x8 af = kf[frag % (K_AHEAD + 1)];
                        const bf16x8 bq = qf[nb][ks];
                        if constexpr (ks == 0) MFMA_32x32x16_INIT(s_nxt[mb][nb], af, bq);
                        else MFMA_32x32x16_ACC(s_nxt[mb][nb], af, bq);
                    } else {
                        constexpr int grp = idx / (NB * DB), d = (idx / NB) % DB, nb = idx % NB;
                        constexpr int mb = grp >> 1, hh = grp & 1;
                        constexpr int frag = idx / NB;  // (grp, d) in issue order
                        // prefetch V_AHEAD fragments ahead with this fragment's first MFMA
                        if constexpr (nb == 0 && frag + V_AHEAD < 4 * DB) {
                            constexpr int f2 = frag + V_AHEAD;
                            vf[f2 % (V_AHEAD + 1)] = load_vfrag(vt_cur, (f2 / DB) >> 1, (f2 / DB) & 1, f2 % DB);
                        }
                        o[d][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[frag % (V_AHEAD + 1)], pb[nb][mb][hh],
                                                                           o[d][nb], 0, 0, 0);
                    }
                    constexpr int a0 = s == 0 ? 0 : sch.atoms_end[s == 0 ? 0 : s - 1];
                    constexpr int a1 = sch.atoms_end[s];
                    static_range<a0, a1>([&](auto K) { atom(K); });
                    __builtin_amdgcn_sched_barrier(0);
                });
            };
            if constexpr (has_next) run(std::type_identity<SchedFull>());
            else run(std::type_identity<SchedLast>());
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) l_part[nb] += lsum[nb][0] + lsum[nb][1];
        };

        if (ntiles > 0) {
            typedef std::integral_constant<int, 0> P0;
            typedef std::integral_constant<int, 1> P1;
            typedef std::integral_constant<bool, true> NX;
            typedef std::integral_constant<bool, false> LAST;
            f32x16 s_a[2][NB], s_b[2][NB];
            wait_vmcnt<0>();
            lds_barrier();
            qk_all(kbuf0, s_a);
            mfma_drain();
            // Tiles in pairs (static buffer parity). With an even tile count the
            // last pair computes one S^T tile too many, from stale LDS data, and
            // discards it: cheaper than a third step variant's registers.
            int t = 0;
            for (; t + 1 < ntiles; t += 2) {
                step(P0(), NX(), t, s_a, s_b);
                step(P1(), NX(), t + 1, s_b, s_a);
            }
            if (t < ntiles) step(P0(), LAST(), t, s_a, s_b);
            mfma_drain();
            // a pair's second step may still be copying (zeros) into LDS: no copy
            // may outlive the workgroup's LDS allocation
            wait_vmcnt<0>();
        }

        // ---- epilogue: normalise and store ----
        // The arguments only the epilogue needs are read again from the kernel
        // argument segment (the empty asm hides that they were read before), so
        // they do not occupy scalar registers across the key loop.
        const AttnArgs* ka = (const AttnArgs*)__builtin_amdgcn_kernarg_segment_ptr();
        asm volatile("" : "+s"(ka));
        const WorkItem it2 = ka->items[item_id];
        const int row0 = __builtin_amdgcn_readfirstlane(it2.row0);
        const int split = __builtin_amdgcn_readfirstlane(it2.split);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const float l_tot = lane_swap32_add(l_part[nb]);
            const float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
            const float lse_val = l_tot > 0.f ? (m_run[nb] + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
            if (!qvalid[nb]) continue;
            const int row = row0 + wave * WROWS + nb * 32 + lr;
            if constexpr (SPLIT) {
                float* po = (float*)ka->out + (((int64_t)split * ka->tokens + row) * ka->num_heads + h) * DV;
#pragma unroll
                for (int d = 0; d < DB; ++d)
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        float4 w = {o[d][nb][c * 4 + 0] * inv_l, o[d][nb][c * 4 + 1] * inv_l,
                                    o[d][nb][c * 4 + 2] * inv_l, o[d][nb][c * 4 + 3] * inv_l};
                        *(float4*)(po + d * 32 + c * 8 + lg * 4) = w;
                    }
                if (lg == 0) ka->lse[((int64_t)split * ka->num_heads + h) * ka->tokens + row] = lse_val;
            } else {
                u16* op = (u16*)ka->out + (int64_t)row * ka->o_st + (int64_t)h * ka->o_sh;
#pragma unroll
                for (int d = 0; d < DB; ++d)
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        bf16x4 w;
#pragma unroll
                        for (int j = 0; j < 4; ++j) w[j] = (__bf16)(o[d][nb][c * 4 + j] * inv_l);
                        *(bf16x4*)(op + d * 32 + c * 8 + lg * 4) = w;
                    }
                if (lg == 0 && ka->lse) ka->lse[(int64_t)h * ka->lse_sh + row] = lse_val;
            }
        }
    }  // slot entries
}


// Merge of split partials: lse = log sum_s exp(lse_s); out = sum_s exp(lse_s - lse) O_s.
template <int DV>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
    constexpr int G = DV / 4;  // threads per (row, head): 4 values each
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t pair = gid / G;
    const int c = (int)(gid % G);
    if (pair >= (int64_t)a.tokens * a.num_heads) return;
    const int row = (int)(pair / a.num_heads);
    const int h = (int)(pair % a.num_heads);
    float ls[MAX_SPLITS];
    float mx = -INFINITY;
    for (int s = 0; s < a.splits; ++s) {
        ls[s] = a.part_lse[((int64_t)s * a.num_heads + h) * a.tokens + row];
        mx = fmaxf(mx, ls[s]);
    }
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int s = 0; s < a.splits; ++s) {
        const float w = (ls[s] == -INFINITY) ? 0.f : __expf(ls[s] - mx);
        den += w;
        const float4 v = *(const float4*)(a.part_o + (((int64_t)s * a.tokens + row) * a.num_heads + h) * DV + c * 4);
        acc[0] += w * v.x;
        acc[1] += w * v.y;
        acc[2] += w * v.z;
        acc[3] += w * v.w;
    }
    const float inv = 1.f / den;
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = (__bf16)(acc[j] * inv);
    *(bf16x4*)(a.out + (int64_t)row * a.o_st + (int64_t)h * a.o_sh + c * 4) = r;
    if (c == 0 && a.lse) a.lse[(int64_t)h * a.lse_sh + row] = mx + __logf(den);
}

[[maybe_unused]] size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <int DQK, int DV, int NB, int KVM>
hipError_t launch(const AttnArgs& a, bool split, const CombineArgs& ca, hipStream_t stream) {
    const int64_t total = (int64_t)a.num_slots * a.num_heads;
    if (total <= 0) return hipSuccess;
    if (total > (int64_t)INT32_MAX) return hipErrorInvalidValue;
    dim3 grid((unsigned)total), block(NTHREADS);
    if (split) {
        hipLaunchKernelGGL((attn_fwd_kernel<DQK, DV, NB, true, KVM>), grid, block, 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t threads = (int64_t)ca.tokens * ca.num_heads * (DV / 4);
        dim3 cg((unsigned)((threads + 255) / 256));
        hipLaunchKernelGGL((combine_kernel<DV>), cg, dim3(256), 0, stream, ca);
    } else {
        hipLaunchKernelGGL((attn_fwd_kernel<DQK, DV, NB, false, KVM>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

template <int KVM>
hipError_t launch_dims(int nb, int dqk, const AttnArgs& a, bool split, const CombineArgs& ca, hipStream_t stream) {
    if constexpr (KVM == KV_ROPE) {
        // the split key layout exists for dqk = 192 only (the caller checks)
        if (nb == 1) return launch<192, 128, 1, KVM>(a, split, ca, stream);
        return launch<192, 128, 2, KVM>(a, split, ca, stream);
    } else {
        if (nb == 1) {
            if (dqk == 64) return launch<64, 64, 1, KVM>(a, split, ca, stream);
            if (dqk == 128) return launch<128, 128, 1, KVM>(a, split, ca, stream);
            return launch<192, 128, 1, KVM>(a, split, ca, stream);
        }
        if (dqk == 64) return launch<64, 64, 2, KVM>(a, split, ca, stream);
        if (dqk == 128) return launch<128, 128, 2, KVM>(a, split, ca, stream);
        return launch<192, 128, 2, KVM>(a, split, ca, stream);
    }
}

}  // namespace

#if VPP_PART == 0 || VPP_PART == 3
hipError_t vpp_detail::launch_attn_contig(int nb, int dqk, const AttnArgs& a, bool split,
                                          const CombineArgs& ca, hipStream_t stream) {
    return launch_dims<KV_CONTIG>(nb, dqk, a, split, ca, stream);
}
#endif
#if VPP_PART == 1 || VPP_PART == 3
hipError_t vpp_detail::launch_attn_paged(int nb, int dqk, const AttnArgs& a, bool split,
                                         const CombineArgs& ca, hipStream_t stream) {
    return launch_dims<KV_PAGED>(nb, dqk, a, split, ca, stream);
}
#endif
#if VPP_PART == 2 || VPP_PART == 3
hipError_t vpp_detail::launch_attn_rope(int nb, const AttnArgs& a, bool split, const CombineArgs& ca,
                                        hipStream_t stream) {
    return launch_dims<KV_ROPE>(nb, 192, a, split, ca, stream);
}
#endif

#if VPP_PART == 0 || VPP_PART == 3

// Scatter of a chunk's new K/V rows into a paged cache: the write that puts a
// chunk's own keys and values in the cache before its attention (section 2.4).
// One thread moves one 16-byte granule; consecutive threads walk the granules
// of one (token, head) row, K first, so reads and writes are contiguous runs.
// slot = page * page_size + row; slots outside [0, num_pages * page_size) are
// skipped (padding tokens use -1).
struct AppendArgs {
    const u16* k_new;
    const u16* v_new;
    u16* k_pages;
    u16* v_pages;
    const int64_t* slots;
    int64_t kn_st, kn_sh, vn_st, vn_sh;  // element strides
    int64_t k_sp, k_st, k_sh, v_sp, v_st, v_sh;
    int32_t tokens, heads, k_gran, v_gran, page_shift, num_pages;
};

__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
    const int per = a.k_gran + a.v_gran;  // granules per (token, head)
    const int gid = (int)(blockIdx.x * 256u + threadIdx.x);
    if (gid >= a.tokens * a.heads * per) return;
    const int g = gid % per;
    const int th = gid / per;
    const int h = th % a.heads;
    const int t = th / a.heads;
    const int64_t slot = a.slots[t];
    if (slot < 0 || slot >= ((int64_t)a.num_pages << a.page_shift)) return;
    const int64_t page = slot >> a.page_shift;
    const int64_t row = slot & (((int64_t)1 << a.page_shift) - 1);
    if (g < a.k_gran) {
        const uint4* src = (const uint4*)(a.k_new + (int64_t)t * a.kn_st + (int64_t)h * a.kn_sh) + g;
        uint4* dst = (uint4*)(a.k_pages + page * a.k_sp + row * a.k_st + (int64_t)h * a.k_sh) + g;
        *dst = *src;
    } else {
        const int gv = g - a.k_gran;
        const uint4* src = (const uint4*)(a.v_new + (int64_t)t * a.vn_st + (int64_t)h * a.vn_sh) + gv;
        uint4* dst = (uint4*)(a.v_pages + page * a.v_sp + row * a.v_st + (int64_t)h * a.v_sh) + gv;
        *dst = *src;
    }
}

// ---------------------------------------------------------------------------
// host side: plan
// ---------------------------------------------------------------------------
struct vpp_chunk_attn_plan_s {
    vpp_chunk_attn_config_t cfg;
    float scale;
    std::vector<WorkItem> items;
    std::vector<int32_t> item_seg;  // segment of each work item (paged runs)
    int32_t num_slots = 0;          // workgroups per head: items.size() / 2
    int32_t num_tiles = 0;
    int32_t num_splits = 1;
    int32_t nb = 2;  // 32-row query blocks per wave of the kernel variant the plan was made for
    int32_t tokens = 0;
    double pairs = 0.0;
    size_t items_bytes = 0;
    size_t ws_bytes = 0;
    // pinned staging ring for the work-list copy, created on first run
    WorkItem* staging[STAGING_SLOTS] = {};
    size_t staging_cap[STAGING_SLOTS] = {};
    hipEvent_t staging_done[STAGING_SLOTS] = {};
    bool staging_pending[STAGING_SLOTS] = {};
    int next_slot = 0;
    int device = -1;
};

namespace {

bool supported_dims(int dqk, int dv) {
    return (dqk == 64 && dv == 64) || (dqk == 128 && dv == 128) || (dqk == 192 && dv == 128);
}

// Kernel variant for a chunk: query blocks of 32 rows per wave. 64-row waves
// (NB = 2) unless the chunk is small and its key ranges short (at most two
// 256-row workgroups per CU, at most 8192 keys per tile on average): there the
// finer 128-row tiles (NB = 1, two workgroups per CU) even out the unequal
// key ranges of the diagonal tiles. With dqk = 192 the 32-row variant runs out
// of registers, so it keeps NB = 2. VPP_NB overrides, for tuning.
int choose_nb(const vpp_chunk_attn_config_t& c, int64_t tiles256, double mean_keys256) {
    const char* e = getenv("VPP_NB");
    if (e && (atoi(e) == 1 || atoi(e) == 2)) return atoi(e);
    if (c.head_dim_qk <= 128 && tiles256 * c.num_q_heads <= 2 * 256 && mean_keys256 <= 8192.0) return 1;
    return 2;
}

vpp_status_t check_config(const vpp_chunk_attn_config_t& c) {
    if (c.num_q_heads <= 0 || c.num_kv_heads <= 0 || c.num_q_heads % c.num_kv_heads != 0)
        return VPP_ERR_INVALID_ARG;
    if (c.max_chunk_tokens <= 0 || c.max_segments <= 0 || c.max_kv_len <= 0) return VPP_ERR_INVALID_ARG;
    if (c.max_kv_len > (int64_t)INT32_MAX - BM_MAX) return VPP_ERR_INVALID_ARG;
    if (!(c.softmax_scale >= 0.f) || !isfinite(c.softmax_scale)) return VPP_ERR_INVALID_ARG;
    if (c.num_splits == 0 || c.num_splits < -1 || c.num_splits > MAX_SPLITS) return VPP_ERR_INVALID_ARG;
    if (c.causal != 1) return VPP_ERR_UNSUPPORTED;
    if (!supported_dims(c.head_dim_qk, c.head_dim_v)) return VPP_ERR_UNSUPPORTED;
    return VPP_OK;
}

// Split count. A split cuts the prefix [0, p) of a segment into n tile-aligned
// parts common to all of its tiles; the last part runs on to each tile's own end
// (its keys within the chunk), so pieces of one index read the same keys in every
// tile. Explicit: the requested count, at most one piece per key tile of the
// longest prefix (a chunk without a prefix is not split). Automatic: the count
// whose launch a model of the hardware's workgroup placement finishes first,
// charging the fp32 partials that a split writes and the merge reads back
// (see auto_split below); pieces hold at least MIN_PIECE prefix keys, and a
// split must be predicted to gain at least 3 %.
constexpr int64_t MIN_PIECE = 1024;
int fixed_splits(const vpp_chunk_attn_config_t& c, int64_t max_prefix) {
    return (int)std::min<int64_t>(c.num_splits, std::max<int64_t>(1, max_prefix / BN));
}

// Boundary b of the n-part split of a p-key prefix (tile-aligned, b = 0 .. n-1).
int32_t piece_begin(int64_t p, int n, int b) { return (int32_t)(((p / BN) * b / n) * BN); }

// Automatic split count: simulate the launch of each candidate count and keep
// the fastest. The grid is slots x heads, head-major, remapped so that XCD x
// runs the x-th eighth of that order (work_coords); each XCD places its
// workgroups in order on whichever of its CU slots frees first (32 CUs, times
// the workgroups a CU holds). A workgroup costs its key tiles plus a fixed
// amount per tile it runs (Q load, pipeline fill, store). A split count n > 1
// also costs the fp32 partials its pieces write and the merge reads back. The
// unsplit plan is kept whenever its simulated makespan is within 5 % of the
// ideal (total work spread evenly), which covers every chunk with enough even
// slots.
template <typename Build>
int auto_split(const vpp_chunk_attn_config_t& c, int bm, int wg_per_cu, int64_t max_prefix, int32_t tokens,
               Build&& build) {
    constexpr int NXCD = 8, CU_PER_XCD = 32;
    constexpr double TILE_OVERHEAD = 2.0;  // fixed cost of a tile, in key tiles
    const int heads = c.num_q_heads;
    // one key tile of one workgroup: 2 bm BN (dqk + dv) flop at ~5 TFLOP/s per CU
    const double tile_s = 2.0 * bm * BN * (c.head_dim_qk + c.head_dim_v) / 5.0e12;
    std::vector<WorkItem> list;
    auto entry_cost = [](const WorkItem& w) {
        return w.nrows ? (double)((w.key_end - w.key_begin + BN - 1) / BN) + TILE_OVERHEAD : 0.0;
    };
    // simulated seconds of the launch, and of its work spread evenly over the chip
    auto simulate = [&](int n, double& ideal) {
        build(n, list);
        const int64_t nslots = (int64_t)list.size() / 2;
        std::vector<double> cost((size_t)nslots);
        double total = 0.0;
        for (int64_t i = 0; i < nslots; ++i) {
            cost[(size_t)i] = entry_cost(list[(size_t)(2 * i)]) + entry_cost(list[(size_t)(2 * i + 1)]);
            total += cost[(size_t)i];
        }
        const int lanes = CU_PER_XCD * wg_per_cu;
        ideal = total * heads / (NXCD * lanes) * tile_s;
        const int64_t all = nslots * heads, per = all / NXCD;
        double makespan = 0.0;
        std::vector<double> free_at;
        // with whole heads per XCD every XCD runs the same sequence: one suffices
        const int xcds = heads % NXCD == 0 ? 1 : NXCD;
        for (int x = 0; x < xcds; ++x) {
            free_at.assign((size_t)lanes, 0.0);  // a min-heap of lane free times
            auto place = [&](int64_t logical) {
                std::pop_heap(free_at.begin(), free_at.end(), std::greater<double>());
                free_at.back() += cost[(size_t)(logical % nslots)];
                std::push_heap(free_at.begin(), free_at.end(), std::greater<double>());
            };
            for (int64_t j = 0; j < per; ++j) place(x * per + j);
            for (int64_t L = per * NXCD + x; L < all; L += NXCD) place(L);  // the part left unremapped
            makespan = std::max(makespan, *std::max_element(free_at.begin(), free_at.end()));
        }
        return makespan * tile_s;
    };
    double ideal1 = 0.0;
    const double t1 = simulate(1, ideal1);
    if (t1 <= 1.05 * ideal1) return 1;
    const int64_t cap = std::min<int64_t>(MAX_SPLITS, max_prefix / MIN_PIECE);
    // partial bytes per piece: fp32 out and lse of every (row, head), written once and
    // read once, at the ~3 TB/s the split chunks of the mixed workload were measured to
    // pay; a split must also be predicted to gain at least 3 %
    const double partial_s = 2.0 * tokens * heads * (4.0 * c.head_dim_v + 4.0) / 3.0e12;
    int best = 1;
    double best_t = 0.97 * t1;
    static const int candidates[] = {2, 3, 4, 6, 8, 12, 16};
    for (int n : candidates) {
        if (n > cap) break;
        double ideal = 0.0;
        const double t = simulate(n, ideal) + n * partial_s;
        if (t < best_t) {
            best_t = t;
            best = n;
        }
    }
    return best;
}

}  // namespace

extern "C" vpp_status_t vpp_chunk_attn_plan(const vpp_chunk_attn_config_t* cfg, int32_t num_segments,
                                            const int32_t* cu_q, const int64_t* kv_start,
                                            const int64_t* prefix_len, vpp_chunk_attn_plan_t* inout_plan,
                                            size_t* workspace_bytes) {
    if (!inout_plan || !workspace_bytes) return VPP_ERR_INVALID_ARG;
    vpp_chunk_attn_plan_s* p = *inout_plan;
    vpp_chunk_attn_config_t c;
    if (p) {
        c = cfg ? *cfg : p->cfg;
        if (cfg && memcmp(cfg, &p->cfg, sizeof c) != 0) return VPP_ERR_INVALID_ARG;
    } else {
        if (!cfg) return VPP_ERR_INVALID_ARG;
        c = *cfg;
    }
    vpp_status_t st = check_config(c);
    if (st != VPP_OK) return st;
    if (num_segments <= 0 || num_segments > c.max_segments) return VPP_ERR_INVALID_ARG;
    if (!cu_q || !kv_start || !prefix_len) return VPP_ERR_INVALID_ARG;
    if (cu_q[0] != 0) return VPP_ERR_INVALID_ARG;
    for (int s = 0; s < num_segments; ++s) {
        if (cu_q[s + 1] < cu_q[s]) return VPP_ERR_INVALID_ARG;
        if (kv_start[s] < 0 || prefix_len[s] < 0) return VPP_ERR_INVALID_ARG;
        const int64_t len = cu_q[s + 1] - cu_q[s];
        if (prefix_len[s] > c.max_kv_len || kv_start[s] > c.max_kv_len) return VPP_ERR_INVALID_ARG;
        if (kv_start[s] + prefix_len[s] + len > c.max_kv_len) return VPP_ERR_INVALID_ARG;
    }
    if (cu_q[num_segments] > c.max_chunk_tokens) return VPP_ERR_INVALID_ARG;

    // query tiles of every segment, with their whole key range [0, last position + 1)
    int64_t tiles256 = 0;
    double keys256 = 0.0;
    for (int s = 0; s < num_segments; ++s)
        for (int r0 = cu_q[s]; r0 < cu_q[s + 1]; r0 += block_rows(2)) {
            ++tiles256;
            keys256 += (double)prefix_len[s] + (r0 - cu_q[s]) + std::min(block_rows(2), cu_q[s + 1] - r0);
        }
    const int nb = choose_nb(c, tiles256, tiles256 ? keys256 / tiles256 : 0.0);
    const int BM = block_rows(nb);
    // Work slots. A workgroup runs one slot: up to two query tiles of one segment,
    // tile i with its key range ascending, then tile T-1-i (the partner from the
    // other end of the segment) descending. A pair's two ranges together span the
    // same number of keys in every slot of the segment, so the workgroups of a
    // segment finish together; and at any moment they all read one of two key
    // positions (the ascending front, and the descending one, which mirrors it), so
    // the tiles running side by side on one XCD share each K/V tile through its L2.
    // Slots are grouped by (segment, split piece); groups run longest first.
    std::vector<WorkItem> items;
    std::vector<int32_t> iseg;
    double pairs = 0.0;
    int ntiles = 0, nsplit = 1;
    try {
        struct Seg { int t0, t1; };  // the segment's tiles in `tiles`
        std::vector<WorkItem> tiles;
        std::vector<Seg> segs((size_t)num_segments);
        int64_t max_prefix = 0;
        for (int s = 0; s < num_segments; ++s) {
            segs[s].t0 = (int)tiles.size();
            for (int r0 = cu_q[s]; r0 < cu_q[s + 1]; r0 += BM) {
                WorkItem w;
                w.row0 = r0;
                w.nrows = std::min(BM, cu_q[s + 1] - r0);
                w.pos0 = (int32_t)(prefix_len[s] + (r0 - cu_q[s]));
                w.key_begin = 0;
                w.key_end = w.pos0 + w.nrows;
                w.split = 0;
                w.kv_base = kv_start[s];
                tiles.push_back(w);
                // visible pairs: sum over rows of (position + 1)
                pairs += (double)w.nrows * (double)w.pos0 + 0.5 * (double)w.nrows * (w.nrows + 1);
            }
            segs[s].t1 = (int)tiles.size();
            if (segs[s].t1 > segs[s].t0) max_prefix = std::max(max_prefix, prefix_len[s]);
        }
        ntiles = (int)tiles.size();

        // the work list for n split pieces: two entries per slot, grouped by
        // (segment, piece), longest group first
        auto build = [&](int n, std::vector<WorkItem>& out, std::vector<int32_t>* out_seg) {
            struct Group { int seg, piece; int64_t len; size_t first, count; };  // slots [first, first+count)
            std::vector<Group> groups;
            std::vector<WorkItem> grouped;  // two items per slot, group by group
            const WorkItem none = {0, 0, 0, 0, 0, 0, 0};
            for (int s = 0; s < num_segments; ++s) {
                const int T = segs[s].t1 - segs[s].t0;
                if (T == 0) continue;
                for (int b = 0; b < n; ++b) {
                    auto piece = [&](int ti) {
                        WorkItem w = tiles[segs[s].t0 + ti];
                        w.split = b;
                        if (n > 1) {
                            w.key_begin = piece_begin(prefix_len[s], n, b);
                            if (b + 1 < n) w.key_end = piece_begin(prefix_len[s], n, b + 1);
                        }
                        return w;
                    };
                    Group g{s, b, 0, grouped.size() / 2, 0};
                    for (int i = 0; i < (T + 1) / 2; ++i) {
                        const WorkItem x = piece(i);
                        const WorkItem y = (T - 1 - i != i) ? piece(T - 1 - i) : none;
                        grouped.push_back(x);
                        grouped.push_back(y);
                        const int64_t len =
                            (int64_t)(x.key_end - x.key_begin) + (y.nrows ? y.key_end - y.key_begin : 0);
                        g.len = std::max(g.len, len);
                        ++g.count;
                    }
                    groups.push_back(g);
                }
            }
            std::stable_sort(groups.begin(), groups.end(),
                             [](const Group& x, const Group& y) { return x.len > y.len; });
            out.clear();
            out.reserve(grouped.size());
            if (out_seg) {
                out_seg->clear();
                out_seg->reserve(grouped.size());
            }
            for (const Group& g : groups)
                for (size_t k = 0; k < 2 * g.count; ++k) {
                    out.push_back(grouped[2 * g.first + k]);
                    if (out_seg) out_seg->push_back(g.seg);
                }
        };
        if (ntiles == 0) {
            nsplit = 1;
        } else if (c.num_splits >= 1) {
            nsplit = fixed_splits(c, max_prefix);
        } else {
            nsplit = auto_split(c, BM, nb == 1 ? 2 : 1, max_prefix, cu_q[num_segments],
                                [&](int n, std::vector<WorkItem>& out) { build(n, out, nullptr); });
        }
        build(nsplit, items, &iseg);
    } catch (const std::bad_alloc&) {
        return VPP_ERR_NOMEM;
    }

    if (!p) {
        p = new (std::nothrow) vpp_chunk_attn_plan_s();
        if (!p) return VPP_ERR_NOMEM;
        p->cfg = c;
        *inout_plan = p;
    }
    p->nb = nb;
    p->scale = c.softmax_scale > 0.f ? c.softmax_scale : (float)(1.0 / sqrt((double)c.head_dim_qk));
    p->items.swap(items);
    p->item_seg.swap(iseg);
    p->num_tiles = ntiles;
    p->num_splits = nsplit;
    p->tokens = cu_q[num_segments];
    p->pairs = pairs;
    p->num_slots = (int32_t)(p->items.size() / 2);
    p->items_bytes = p->items.size() * sizeof(WorkItem);
    size_t ws = align256(std::max<size_t>(p->items_bytes, 1));
    if (nsplit > 1) {
        ws += align256((size_t)nsplit * p->tokens * c.num_q_heads * c.head_dim_v * sizeof(float));
        ws += align256((size_t)nsplit * c.num_q_heads * p->tokens * sizeof(float));
    }
    p->ws_bytes = ws;
    *workspace_bytes = ws;
    return VPP_OK;
}

extern "C" vpp_status_t vpp_chunk_attn_plan_info(vpp_chunk_attn_plan_t p, vpp_chunk_attn_plan_info_t* info) {
    if (!p || !info) return VPP_ERR_INVALID_ARG;
    info->num_tiles = p->num_tiles;
    info->num_splits = p->num_splits;
    info->num_work_items = (int32_t)p->items.size();
    info->num_slots = p->num_slots;
    info->block_m = block_rows(p->nb);
    info->block_n = BN;
    info->num_tokens = p->tokens;
    info->workspace_bytes = (int64_t)p->ws_bytes;
    info->pairs = p->pairs;
    return VPP_OK;
}

extern "C" vpp_status_t vpp_chunk_attn_plan_items(vpp_chunk_attn_plan_t p, vpp_chunk_attn_work_item_t* items,
                                                  int32_t capacity, int32_t* count) {
    if (!p || !count || capacity < 0 || (capacity > 0 && !items)) return VPP_ERR_INVALID_ARG;
    *count = (int32_t)p->items.size();
    const int32_t n = std::min(capacity, *count);
    if (n > 0) memcpy(items, p->items.data(), sizeof(WorkItem) * (size_t)n);
    return VPP_OK;
}

extern "C" void vpp_chunk_attn_destroy(vpp_chunk_attn_plan_t p) {
    if (!p) return;
    for (int i = 0; i < STAGING_SLOTS; ++i) {
        if (p->staging_done[i]) {
            if (p->staging_pending[i]) (void)hipEventSynchronize(p->staging_done[i]);
            (void)hipEventDestroy(p->staging_done[i]);
        }
        if (p->staging[i]) (void)hipHostFree(p->staging[i]);
    }
    delete p;
}

extern "C" const char* vpp_status_str(vpp_status_t s) {
    switch (s) {
        case VPP_OK: return "ok";
        case VPP_ERR_INVALID_ARG: return "invalid argument";
        case VPP_ERR_UNSUPPORTED: return "unsupported configuration";
        case VPP_ERR_WORKSPACE: return "workspace too small";
        case VPP_ERR_HIP: return "HIP runtime error";
        case VPP_ERR_NOMEM: return "out of host memory";
    }
    return "unknown status";
}

// ---------------------------------------------------------------------------
// host side: run
// ---------------------------------------------------------------------------
namespace {

bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }
bool stride_ok(int64_t s) { return s > 0 && (s % 8) == 0; }

int env_xcd_remap() {
    const char* s = getenv("VPP_XCD_REMAP");
    return s ? atoi(s) : 1;
}

}  // namespace

namespace {

// Paged-cache description of one run (see vpp_chunk_attn_run_paged).
struct PagedKV {
    const int32_t* block_table;
    int64_t bt_st, k_sp, v_sp;
    int32_t page_shift, num_pages;
};

// Shared key part of the split key layout (see vpp_chunk_attn_run_mla).
struct RopeK {
    const void* k_rope;
    int64_t kr_st;
};

// How run_impl puts the work list into the workspace: through the plan's pinned
// staging ring (asynchronous), or straight from the plan's host copy, which
// allocates nothing (the copy out of host memory completes before the call
// returns).
enum class Upload { staged, direct };

vpp_status_t run_impl(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st, int64_t q_sh, const void* k,
                      int64_t k_st, int64_t k_sh, const void* v, int64_t v_st, int64_t v_sh, void* out,
                      int64_t o_st, int64_t o_sh, float* lse, int64_t lse_sh, void* workspace,
                      size_t workspace_bytes, void* stream_ptr, const PagedKV* pg, const RopeK* rope = nullptr,
                      Upload upload = Upload::staged) {
    if (!p) return VPP_ERR_INVALID_ARG;
    if (!q || !k || !v || !out) return VPP_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return VPP_ERR_INVALID_ARG;
    if (!stride_ok(q_st) || !stride_ok(q_sh) || !stride_ok(k_st) || !stride_ok(k_sh) || !stride_ok(v_st) ||
        !stride_ok(v_sh) || !stride_ok(o_st) || !stride_ok(o_sh))
        return VPP_ERR_INVALID_ARG;
    if (lse && (((uintptr_t)lse & 3u) != 0 || lse_sh < p->tokens)) return VPP_ERR_INVALID_ARG;
    // the kernels keep element strides in 32 bits; the bytes of one key tile
    // (BN rows of a cache row stride, 2 bytes an element) must also stay below
    // 2^31, the range of a buffer resource's size field
    const int64_t smax = ((int64_t)1 << 31) / 64;
    const int64_t row_smax = ((int64_t)1 << 31) / (2 * BN);
    if (q_st >= smax || q_sh >= smax || k_st >= row_smax || k_sh >= smax || v_st >= row_smax ||
        v_sh >= smax || o_st >= smax || o_sh >= smax || (lse && lse_sh >= ((int64_t)1 << 31)))
        return VPP_ERR_INVALID_ARG;
    if (rope) {
        if (p->cfg.head_dim_qk != 192 || p->cfg.head_dim_v != 128) return VPP_ERR_UNSUPPORTED;
        if (!rope->k_rope || !aligned16(rope->k_rope) || !stride_ok(rope->kr_st) || rope->kr_st < 64 ||
            rope->kr_st >= row_smax)
            return VPP_ERR_INVALID_ARG;
    }
    if (!workspace || ((uintptr_t)workspace & 255u) != 0) return VPP_ERR_WORKSPACE;
    if (workspace_bytes < p->ws_bytes) return VPP_ERR_WORKSPACE;
    if (p->items.empty()) return VPP_OK;  // nothing to do: every segment is empty

    hipStream_t stream = (hipStream_t)stream_ptr;
    char* ws = (char*)workspace;
    if (upload == Upload::direct) {
        // the paged path rewrites kv_base in its copy of the list; it always stages
        if (pg) return VPP_ERR_INVALID_ARG;
        if (hipMemcpyAsync(ws, p->items.data(), p->items_bytes, hipMemcpyHostToDevice, stream) != hipSuccess)
            return VPP_ERR_HIP;
    } else {
        const int slot = p->next_slot;
        p->next_slot = (p->next_slot + 1) % STAGING_SLOTS;
        if (!p->staging_done[slot]) {
            if (hipEventCreateWithFlags(&p->staging_done[slot], hipEventDisableTiming) != hipSuccess)
                return VPP_ERR_HIP;
        }
        if (p->staging_pending[slot]) {
            if (hipEventSynchronize(p->staging_done[slot]) != hipSuccess) return VPP_ERR_HIP;
            p->staging_pending[slot] = false;
        }
        if (p->staging_cap[slot] < p->items_bytes) {
            if (p->staging[slot]) (void)hipHostFree(p->staging[slot]);
            p->staging[slot] = nullptr;
            p->staging_cap[slot] = 0;
            if (hipHostMalloc((void**)&p->staging[slot], p->items_bytes, hipHostMallocDefault) != hipSuccess)
                return VPP_ERR_HIP;
            p->staging_cap[slot] = p->items_bytes;
        }
        memcpy(p->staging[slot], p->items.data(), p->items_bytes);
        if (pg) {
            // paged: the kernel finds the segment's block-table row from kv_base
            for (size_t i = 0; i < p->items.size(); ++i)
                p->staging[slot][i].kv_base = ((int64_t)p->item_seg[i] << 32) | p->items[i].kv_base;
        }
        if (hipMemcpyAsync(ws, p->staging[slot], p->items_bytes, hipMemcpyHostToDevice, stream) != hipSuccess)
            return VPP_ERR_HIP;
        if (hipEventRecord(p->staging_done[slot], stream) != hipSuccess) return VPP_ERR_HIP;
        p->staging_pending[slot] = true;
    }

    const vpp_chunk_attn_config_t& c = p->cfg;
    AttnArgs a;
    memset(&a, 0, sizeof a);
    a.items = (const WorkItem*)ws;
    a.q = (const u16*)q;
    a.k = (const u16*)k;
    a.v = (const u16*)v;
    a.out = out;
    a.lse = lse;
    a.q_st = (int32_t)q_st; a.q_sh = (int32_t)q_sh; a.k_st = (int32_t)k_st; a.k_sh = (int32_t)k_sh;
    a.v_st = (int32_t)v_st; a.v_sh = (int32_t)v_sh; a.o_st = (int32_t)o_st; a.o_sh = (int32_t)o_sh;
    a.lse_sh = (int32_t)lse_sh;
    // one workgroup per slot and head: the kernel reads entries 2*slot and 2*slot + 1
    a.num_slots = p->num_slots;
    a.num_entries = (int32_t)p->items.size();
    a.num_heads = c.num_q_heads;
    a.group = c.num_q_heads / c.num_kv_heads;
    a.tokens = p->tokens;
    a.scale_log2 = (float)((double)p->scale * 1.4426950408889634);
    a.xcd_remap = env_xcd_remap();
    if (rope) {
        a.k_rope = (const u16*)rope->k_rope;
        a.kr_st = (int32_t)rope->kr_st;
    }
    if (pg) {
        a.block_table = pg->block_table;
        a.bt_st = pg->bt_st;
        a.k_sp = pg->k_sp;
        a.v_sp = pg->v_sp;
        a.page_shift = pg->page_shift;
        a.num_pages = pg->num_pages;
    }
    const bool split = p->num_splits > 1;
    CombineArgs ca;
    memset(&ca, 0, sizeof ca);
    if (split) {
        size_t off = align256(p->items_bytes);
        ca.part_o = (float*)(ws + off);
        off += align256((size_t)p->num_splits * p->tokens * c.num_q_heads * c.head_dim_v * sizeof(float));
        ca.part_lse = (float*)(ws + off);
        a.out = (void*)ca.part_o;
        a.lse = (float*)ca.part_lse;
        ca.out = (u16*)out;
        ca.lse = lse;
        ca.o_st = o_st; ca.o_sh = o_sh; ca.lse_sh = lse_sh;
        ca.tokens = p->tokens;
        ca.num_heads = c.num_q_heads;
        ca.splits = p->num_splits;
    }
    const hipError_t e = rope ? vpp_detail::launch_attn_rope(p->nb, a, split, ca, stream)
                         : pg ? vpp_detail::launch_attn_paged(p->nb, c.head_dim_qk, a, split, ca, stream)
                              : vpp_detail::launch_attn_contig(p->nb, c.head_dim_qk, a, split, ca, stream);
    return e == hipSuccess ? VPP_OK : VPP_ERR_HIP;
}

}  // namespace

extern "C" vpp_status_t vpp_chunk_attn_run(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st, int64_t q_sh,
                                           const void* k, int64_t k_st, int64_t k_sh, const void* v,
                                           int64_t v_st, int64_t v_sh, void* out, int64_t o_st, int64_t o_sh,
                                           float* lse, int64_t lse_sh, void* workspace, size_t workspace_bytes,
                                           void* stream_ptr) {
    return run_impl(p, q, q_st, q_sh, k, k_st, k_sh, v, v_st, v_sh, out, o_st, o_sh, lse, lse_sh, workspace,
                    workspace_bytes, stream_ptr, nullptr);
}

// ---------------------------------------------------------------------------
// No-allocation entry point. Its workspace is this file-scope device array (one
// copy per GPU, held until the process ends). In host code the name `scratch`
// is only a stand-in for the symbol, never a device address: the array's
// address on each device is looked up once, with that device current, and kept.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[VPP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_addr[MAX_DEVICES] = {};

// The current device's copy of `scratch` (looked up on the first call on that device).
vpp_status_t scratch_on_current_device(void** addr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return VPP_ERR_HIP;
    if (dev >= MAX_DEVICES) return VPP_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_addr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return VPP_ERR_HIP;
        scratch_addr[dev] = ptr;
    }
    *addr = scratch_addr[dev];
    return VPP_OK;
}

}  // namespace

extern "C" vpp_status_t vpp_chunk_attn_run_noalloc(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st,
                                                   int64_t q_sh, const void* k, int64_t k_st, int64_t k_sh,
                                                   const void* v, int64_t v_st, int64_t v_sh, void* out,
                                                   int64_t o_st, int64_t o_sh, float* lse, int64_t lse_sh,
                                                   void* stream_ptr) {
    if (!p) return VPP_ERR_INVALID_ARG;
    if (p->ws_bytes > (size_t)VPP_NOALLOC_SCRATCH_BYTES) return VPP_ERR_WORKSPACE;
    void* ws = nullptr;
    const vpp_status_t st = scratch_on_current_device(&ws);
    if (st != VPP_OK) return st;
    return run_impl(p, q, q_st, q_sh, k, k_st, k_sh, v, v_st, v_sh, out, o_st, o_sh, lse, lse_sh, ws,
                    (size_t)VPP_NOALLOC_SCRATCH_BYTES, stream_ptr, nullptr, nullptr, Upload::direct);
}

extern "C" vpp_status_t vpp_chunk_attn_run_mla(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st,
                                               int64_t q_sh, const void* k_nope, int64_t kn_st, int64_t kn_sh,
                                               const void* k_rope, int64_t kr_st, const void* v, int64_t v_st,
                                               int64_t v_sh, void* out, int64_t o_st, int64_t o_sh, float* lse,
                                               int64_t lse_sh, void* workspace, size_t workspace_bytes,
                                               void* stream_ptr) {
    RopeK rope{k_rope, kr_st};
    return run_impl(p, q, q_st, q_sh, k_nope, kn_st, kn_sh, v, v_st, v_sh, out, o_st, o_sh, lse, lse_sh,
                    workspace, workspace_bytes, stream_ptr, nullptr, &rope);
}

extern "C" vpp_status_t vpp_chunk_attn_run_paged(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st,
                                                 int64_t q_sh, const void* k_pages, int64_t k_sp, int64_t k_st,
                                                 int64_t k_sh, const void* v_pages, int64_t v_sp, int64_t v_st,
                                                 int64_t v_sh, int32_t page_size, int32_t num_pages,
                                                 const int32_t* block_table, int64_t bt_st, void* out,
                                                 int64_t o_st, int64_t o_sh, float* lse, int64_t lse_sh,
                                                 void* workspace, size_t workspace_bytes, void* stream_ptr) {
    if (!p || !block_table || ((uintptr_t)block_table & 3u) != 0) return VPP_ERR_INVALID_ARG;
    if (page_size < BN || page_size > (1 << 20) || (page_size & (page_size - 1)) != 0) return VPP_ERR_INVALID_ARG;
    if (num_pages < 1 || bt_st < 0) return VPP_ERR_INVALID_ARG;
    // pages start on 16-byte boundaries, and one page's rows fit the kernels' 32-bit row offsets
    if (!stride_ok(k_sp) || !stride_ok(v_sp) || k_sp < 1 || v_sp < 1) return VPP_ERR_INVALID_ARG;
    if ((int64_t)page_size * k_st >= ((int64_t)1 << 31) || (int64_t)page_size * v_st >= ((int64_t)1 << 31))
        return VPP_ERR_INVALID_ARG;
    for (size_t i = 0; i < p->items.size(); ++i)
        if (p->items[i].kv_base % BN != 0 || p->items[i].kv_base >= ((int64_t)1 << 31))
            return VPP_ERR_INVALID_ARG;  // a key tile must not straddle two pages
    int shift = 0;
    while ((1 << shift) < page_size) ++shift;
    PagedKV pg{block_table, bt_st, k_sp, v_sp, shift, num_pages};
    return run_impl(p, q, q_st, q_sh, k_pages, k_st, k_sh, v_pages, v_st, v_sh, out, o_st, o_sh, lse, lse_sh,
                    workspace, workspace_bytes, stream_ptr, &pg);
}

extern "C" vpp_status_t vpp_kv_append_paged(const void* k_new, int64_t kn_st, int64_t kn_sh, const void* v_new,
                                            int64_t vn_st, int64_t vn_sh, void* k_pages, int64_t k_sp,
                                            int64_t k_st, int64_t k_sh, void* v_pages, int64_t v_sp, int64_t v_st,
                                            int64_t v_sh, int32_t num_tokens, int32_t num_kv_heads,
                                            int32_t head_dim_qk, int32_t head_dim_v, int32_t page_size,
                                            int32_t num_pages, const int64_t* slot_mapping, void* stream_ptr) {
    if (num_tokens < 0 || num_kv_heads < 1 || num_pages < 1) return VPP_ERR_INVALID_ARG;
    if (head_dim_qk < 8 || head_dim_v < 8 || head_dim_qk % 8 || head_dim_v % 8 || head_dim_qk > 1024 ||
        head_dim_v > 1024)
        return VPP_ERR_INVALID_ARG;
    if (page_size < BN || page_size > (1 << 20) || (page_size & (page_size - 1)) != 0) return VPP_ERR_INVALID_ARG;
    if (num_tokens == 0) return VPP_OK;
    if (!k_new || !v_new || !k_pages || !v_pages || !slot_mapping) return VPP_ERR_INVALID_ARG;
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pages) || !aligned16(v_pages) ||
        ((uintptr_t)slot_mapping & 7u) != 0)
        return VPP_ERR_INVALID_ARG;
    const int64_t st[] = {kn_st, kn_sh, vn_st, vn_sh, k_sp, k_st, k_sh, v_sp, v_st, v_sh};
    for (int64_t x : st)
        if (!stride_ok(x)) return VPP_ERR_INVALID_ARG;
    const int64_t total = (int64_t)num_tokens * num_kv_heads * ((head_dim_qk + head_dim_v) / 8);
    if (total >= ((int64_t)1 << 31) - 256) return VPP_ERR_INVALID_ARG;
    AppendArgs a;
    a.k_new = (const u16*)k_new;
    a.v_new = (const u16*)v_new;
    a.k_pages = (u16*)k_pages;
    a.v_pages = (u16*)v_pages;
    a.slots = slot_mapping;
    a.kn_st = kn_st; a.kn_sh = kn_sh; a.vn_st = vn_st; a.vn_sh = vn_sh;
    a.k_sp = k_sp; a.k_st = k_st; a.k_sh = k_sh; a.v_sp = v_sp; a.v_st = v_st; a.v_sh = v_sh;
    a.tokens = num_tokens;
    a.heads = num_kv_heads;
    a.k_gran = head_dim_qk / 8;
    a.v_gran = head_dim_v / 8;
    int shift = 0;
    while ((1 << shift) < page_size) ++shift;
    a.page_shift = shift;
    a.num_pages = num_pages;
    hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                       (hipStream_t)stream_ptr, a);
    return hipGetLastError() == hipSuccess ? VPP_OK : VPP_ERR_HIP;
}

extern "C" vpp_status_t vpp_paged_slot_mapping(int32_t num_segments, const int32_t* cu_q, const int64_t* kv_start,
                                               const int64_t* prefix_len, const int32_t* block_table,
                                               int64_t block_table_stride, int32_t pages_per_row,
                                               int32_t page_size, int64_t* slot_mapping) {
    if (num_segments < 0 || !cu_q || page_size < 1 || pages_per_row < 0 || block_table_stride < 0)
        return VPP_ERR_INVALID_ARG;
    if (num_segments == 0) return VPP_OK;
    if (!kv_start || !prefix_len || !block_table || !slot_mapping || cu_q[0] != 0) return VPP_ERR_INVALID_ARG;
    for (int s = 0; s < num_segments; ++s) {
        if (cu_q[s + 1] < cu_q[s] || kv_start[s] < 0 || prefix_len[s] < 0) return VPP_ERR_INVALID_ARG;
        for (int r = cu_q[s]; r < cu_q[s + 1]; ++r) {
            const int64_t row = kv_start[s] + prefix_len[s] + (r - cu_q[s]);
            const int64_t idx = row / page_size;
            if (idx >= pages_per_row) return VPP_ERR_INVALID_ARG;
            const int32_t pg = block_table[(int64_t)s * block_table_stride + idx];
            if (pg < 0) return VPP_ERR_INVALID_ARG;
            slot_mapping[r] = (int64_t)pg * page_size + row % page_size;
        }
    }
    return VPP_OK;
}

#endif  // host code (part 0)

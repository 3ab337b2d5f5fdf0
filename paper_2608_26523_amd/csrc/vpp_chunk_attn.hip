// vpp_chunk_attn.hip -- chunked-prefill causal attention for MI355X (gfx950).
//
// Computes Eq. (1) of the paper (section 2.1), softmax(Q K^T * scale) V under
// the causal rule, for one chunk of query tokens at in-request positions
// prefix .. prefix+len-1 attending to the cached prefix plus the chunk itself
// (section 2.4). Several requests may share a chunk (packing, section 5.3).
//
// Kernel layout (one workgroup = 4 waves = one tile of 128 query rows of one
// query head; keys stream through LDS 64 at a time):
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: keys are the M dimension,
//     queries the N dimension, head dim the K dimension. Each lane then owns
//     one query (column lane%32) and 16 keys per 32-key block, so a row max or
//     row sum needs only one exchange with lane^32.
//   * Online softmax in fp32 with exp2 (scale folded with log2 e).
//   * O^T = V^T P^T on the same MFMA: P leaves the S^T accumulators already in
//     the B-operand layout (no shuffles); V is staged transposed in LDS so that
//     each lane reads its 8 keys of one value column with two 8-byte reads.
//   * Only key tiles that cross the diagonal (or the end of the key range) are
//     masked; tiles past a wave's last query are skipped by that wave.
//   * Split-KV: a tile's key range may be cut into pieces whose fp32 partial
//     results are merged by their log-sum-exp in a second pass.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

#include "vpp_chunk_attn.h"

namespace {

constexpr int BM = 128;        // query rows per workgroup tile
constexpr int BN = 64;         // keys per inner step
constexpr int NTHREADS = 256;  // 4 waves of 64
constexpr int MAX_SPLITS = 16;
constexpr int STAGING_SLOTS = 4;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16;

typedef vpp_chunk_attn_work_item_t WorkItem;
static_assert(sizeof(WorkItem) == 32, "work item layout");

struct AttnArgs {
    const WorkItem* items;
    const u16* q;
    const u16* k;
    const u16* v;
    u16* out;
    float* lse;
    float* part_o;    // split mode: [splits][tokens][Hq][DV] fp32
    float* part_lse;  // split mode: [splits][Hq][tokens] fp32
    int64_t q_st, q_sh, k_st, k_sh, v_st, v_sh, o_st, o_sh, lse_sh;
    int32_t num_items;
    int32_t num_heads;
    int32_t group;     // Hq / Hkv
    int32_t tokens;    // chunk rows (partial layout)
    float scale_log2;  // softmax scale * log2(e)
    int32_t xcd_remap;
};

template <int DQK, int DV>
struct Smem {
    static constexpr int K_STRIDE = DQK + 8;  // 16-byte pad: conflict-free 16 B row reads
    static constexpr int VT_STRIDE = BN + 4;  // 8-byte pad: conflict-free 8 B column reads
    u16 k[BN * K_STRIDE];
    u16 vt[DV * VT_STRIDE];
};

__device__ __forceinline__ float wave_swap32_max(float x) {
    return fmaxf(x, __shfl_xor(x, 32, 64));
}
__device__ __forceinline__ float wave_swap32_add(float x) {
    return x + __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ uint32_t half16(const u32x4& r, int c) {
    return (r[c >> 1] >> ((c & 1) * 16)) & 0xFFFFu;
}

// Launch-order index -> (item, head). With remapping on, the hardware's
// round-robin placement of consecutive workgroups on the 8 XCDs is undone so
// that each XCD runs a contiguous run of logical work (the tiles of the same
// heads, which read the same K/V through that XCD's L2).
__device__ __forceinline__ void work_coords(const AttnArgs& a, int& item, int& head) {
    const int64_t total = (int64_t)a.num_items * a.num_heads;
    int64_t L = blockIdx.x;
    if (a.xcd_remap) {
        const int64_t per = total / 8;
        if (L < per * 8) L = (L % 8) * per + L / 8;
    }
    head = (int)(L / a.num_items);
    item = (int)(L % a.num_items);
}

template <int DQK, int DV, bool SPLIT>
__global__ __launch_bounds__(NTHREADS) void attn_fwd_kernel(AttnArgs a) {
    __shared__ Smem<DQK, DV> sm;
    constexpr int KS = DQK / 16;   // MFMA k-steps for S
    constexpr int DB = DV / 32;    // 32-wide value blocks
    constexpr int K_STRIDE = Smem<DQK, DV>::K_STRIDE;
    constexpr int VT_STRIDE = Smem<DQK, DV>::VT_STRIDE;

    int item_id, h;
    work_coords(a, item_id, h);
    const WorkItem it = a.items[item_id];
    const int hk = h / a.group;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lr = lane & 31;
    const int lg = lane >> 5;

    // This lane's query row: B-operand fragments of Q in registers.
    const int rloc = wave * 32 + lr;
    const bool row_valid = rloc < it.nrows;
    const int qpos = it.pos0 + rloc;
    bf16x8 qf[KS];
    {
        const u16* qp = a.q + (int64_t)(it.row0 + (row_valid ? rloc : 0)) * a.q_st + (int64_t)h * a.q_sh;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            u32x4 raw = {0u, 0u, 0u, 0u};
            if (row_valid) raw = *(const u32x4*)(qp + ks * 16 + lg * 8);
            qf[ks] = __builtin_bit_cast(bf16x8, raw);
        }
    }
    // last valid query position held by this wave (waves past nrows: none)
    const int wave_rows = min(32, it.nrows - wave * 32);
    const int wave_pos_last = it.pos0 + wave * 32 + wave_rows - 1;
    const int wave_pos_first = it.pos0 + wave * 32;

    float m_run = -INFINITY;  // running max of scaled scores (log2 units)
    float l_run = 0.f;        // this lane's share of the softmax denominator
    f32x16 o[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[d][i] = 0.f;

    const int kb = it.key_begin, ke = it.key_end;
    const u16* kbase = a.k + it.kv_base * a.k_st + (int64_t)hk * a.k_sh;
    const u16* vbase = a.v + it.kv_base * a.v_st + (int64_t)hk * a.v_sh;

    for (int kt = kb; kt < ke; kt += BN) {
        __syncthreads();  // everyone is done reading the previous tile
        // K tile: rows kt..kt+63 -> LDS row-major (zero past the key range)
        for (int e = tid; e < BN * (DQK / 8); e += NTHREADS) {
            const int r = e / (DQK / 8), c = e % (DQK / 8);
            u32x4 val = {0u, 0u, 0u, 0u};
            if (kt + r < ke) val = *(const u32x4*)(kbase + (int64_t)(kt + r) * a.k_st + c * 8);
            *(u32x4*)(&sm.k[r * K_STRIDE + c * 8]) = val;
        }
        // V tile -> LDS transposed: each thread moves 4 keys x 8 value columns
        for (int e = tid; e < (BN / 4) * (DV / 8); e += NTHREADS) {
            const int dg = e % (DV / 8), kg = e / (DV / 8);
            u32x4 r[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int key = kt + kg * 4 + j;
                r[j] = u32x4{0u, 0u, 0u, 0u};
                if (key < ke) r[j] = *(const u32x4*)(vbase + (int64_t)key * a.v_st + dg * 8);
            }
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                u32x2 w;
                w[0] = half16(r[0], c) | (half16(r[1], c) << 16);
                w[1] = half16(r[2], c) | (half16(r[3], c) << 16);
                *(u32x2*)(&sm.vt[(dg * 8 + c) * VT_STRIDE + kg * 4]) = w;
            }
        }
        __syncthreads();

        if (kt > wave_pos_last) continue;  // every key of this tile is after this wave's queries

        // S^T = K Q^T for 64 keys x 32 queries
        f32x16 s[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
            for (int i = 0; i < 16; ++i) s[mb][i] = 0.f;
            const u16* krow = &sm.k[(mb * 32 + lr) * K_STRIDE + lg * 8];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 af = __builtin_bit_cast(bf16x8, *(const u32x4*)(krow + ks * 16));
                s[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, qf[ks], s[mb], 0, 0, 0);
            }
        }

        // scale, mask, running max
        const bool need_mask = (kt + BN - 1 > wave_pos_first) || (kt + BN > ke);
        float mloc = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float t = s[mb][i] * a.scale_log2;
                if (need_mask) {
                    const int kpos = kt + mb * 32 + (i >> 2) * 8 + lg * 4 + (i & 3);
                    if (kpos > qpos || kpos >= ke) t = -INFINITY;
                }
                s[mb][i] = t;
                mloc = fmaxf(mloc, t);
            }
        mloc = wave_swap32_max(mloc);
        const float m_new = fmaxf(m_run, mloc);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        m_run = m_new;

        // P = exp2(t - m), its row sum, and P in bf16 as the B operand of O^T += V^T P^T
        float psum = 0.f;
        bf16x8 pb[2][2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = __builtin_amdgcn_exp2f(s[mb][i] - m_use);
                psum += p;
                pb[mb][i >> 3][i & 7] = (__bf16)p;
            }
        l_run = l_run * alpha + psum;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[d][i] *= alpha;

#pragma unroll
        for (int d = 0; d < DB; ++d) {
            const u16* vrow = &sm.vt[(d * 32 + lr) * VT_STRIDE + lg * 4];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int ko = mb * 32 + hh * 16;
                    const u32x2 lo = *(const u32x2*)(vrow + ko);
                    const u32x2 hi = *(const u32x2*)(vrow + ko + 8);
                    const u32x4 raw = {lo[0], lo[1], hi[0], hi[1]};
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, raw), pb[mb][hh], o[d], 0, 0, 0);
                }
        }
    }

    // epilogue: normalise and store
    const float l_tot = wave_swap32_add(l_run);
    const float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse_val = l_tot > 0.f ? (m_run + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
    if (!row_valid) return;
    const int row = it.row0 + rloc;
    if constexpr (SPLIT) {
        float* po = a.part_o + (((int64_t)it.split * a.tokens + row) * a.num_heads + h) * DV;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                float4 w = {o[d][c * 4 + 0] * inv_l, o[d][c * 4 + 1] * inv_l,
                            o[d][c * 4 + 2] * inv_l, o[d][c * 4 + 3] * inv_l};
                *(float4*)(po + d * 32 + c * 8 + lg * 4) = w;
            }
        if (lg == 0) a.part_lse[((int64_t)it.split * a.num_heads + h) * a.tokens + row] = lse_val;
    } else {
        u16* op = a.out + (int64_t)row * a.o_st + (int64_t)h * a.o_sh;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                bf16x4 w;
#pragma unroll
                for (int j = 0; j < 4; ++j) w[j] = (__bf16)(o[d][c * 4 + j] * inv_l);
                *(bf16x4*)(op + d * 32 + c * 8 + lg * 4) = w;
            }
        if (lg == 0 && a.lse) a.lse[(int64_t)h * a.lse_sh + row] = lse_val;
    }
}

// Merge of split partials: lse = log sum_s exp(lse_s); out = sum_s exp(lse_s - lse) O_s.
struct CombineArgs {
    const float* part_o;
    const float* part_lse;
    u16* out;
    float* lse;
    int64_t o_st, o_sh, lse_sh;
    int32_t tokens, num_heads, splits;
};

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

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

// ---------------------------------------------------------------------------
// host side: plan
// ---------------------------------------------------------------------------
struct vpp_chunk_attn_plan_s {
    vpp_chunk_attn_config_t cfg;
    float scale;
    std::vector<WorkItem> items;
    int32_t num_tiles = 0;
    int32_t num_splits = 1;
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

vpp_status_t check_config(const vpp_chunk_attn_config_t& c) {
    if (c.num_q_heads <= 0 || c.num_kv_heads <= 0 || c.num_q_heads % c.num_kv_heads != 0)
        return VPP_ERR_INVALID_ARG;
    if (c.max_chunk_tokens <= 0 || c.max_segments <= 0 || c.max_kv_len <= 0) return VPP_ERR_INVALID_ARG;
    if (c.max_kv_len > (int64_t)INT32_MAX - BM) return VPP_ERR_INVALID_ARG;
    if (!(c.softmax_scale >= 0.f) || !isfinite(c.softmax_scale)) return VPP_ERR_INVALID_ARG;
    if (c.num_splits == 0 || c.num_splits < -1 || c.num_splits > MAX_SPLITS) return VPP_ERR_INVALID_ARG;
    if (c.causal != 1) return VPP_ERR_UNSUPPORTED;
    if (!supported_dims(c.head_dim_qk, c.head_dim_v)) return VPP_ERR_UNSUPPORTED;
    return VPP_OK;
}

// Split count: explicit, or automatic -- split only when the chunk gives too
// few workgroups to fill the chip and the key ranges are long enough that each
// piece still streams many key tiles.
int choose_splits(const vpp_chunk_attn_config_t& c, int tiles, double mean_key_tiles) {
    if (c.num_splits >= 1) return c.num_splits;
    const double wgs = (double)tiles * c.num_q_heads;
    const double target = 2.0 * 256.0;
    if (wgs >= target) return 1;
    int n = (int)ceil(target / std::max(1.0, wgs));
    n = std::min(n, (int)(mean_key_tiles / 8.0));
    return std::max(1, std::min(n, MAX_SPLITS));
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
    std::vector<WorkItem> tiles;
    double pairs = 0.0, key_tiles = 0.0;
    try {
        for (int s = 0; s < num_segments; ++s) {
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
                key_tiles += ceil((double)w.key_end / BN);
            }
        }
    } catch (const std::bad_alloc&) {
        return VPP_ERR_NOMEM;
    }
    const int ntiles = (int)tiles.size();
    const int nsplit = ntiles ? choose_splits(c, ntiles, key_tiles / ntiles) : 1;

    std::vector<WorkItem> items;
    try {
        items.reserve((size_t)ntiles * nsplit);
        for (const WorkItem& t : tiles) {
            const int nkt = (t.key_end + BN - 1) / BN;
            for (int sp = 0; sp < nsplit; ++sp) {
                WorkItem w = t;
                w.split = sp;
                if (nsplit > 1) {
                    w.key_begin = (int32_t)((int64_t)nkt * sp / nsplit) * BN;
                    w.key_end = sp + 1 == nsplit ? t.key_end : (int32_t)((int64_t)nkt * (sp + 1) / nsplit) * BN;
                    w.key_end = std::min(w.key_end, t.key_end);
                    w.key_begin = std::min(w.key_begin, w.key_end);
                }
                items.push_back(w);
            }
        }
    } catch (const std::bad_alloc&) {
        return VPP_ERR_NOMEM;
    }
    // longest key range first, so the short ones fill the tail of the launch
    std::stable_sort(items.begin(), items.end(), [](const WorkItem& x, const WorkItem& y) {
        return (x.key_end - x.key_begin) > (y.key_end - y.key_begin);
    });

    if (!p) {
        p = new (std::nothrow) vpp_chunk_attn_plan_s();
        if (!p) return VPP_ERR_NOMEM;
        p->cfg = c;
        *inout_plan = p;
    }
    p->scale = c.softmax_scale > 0.f ? c.softmax_scale : (float)(1.0 / sqrt((double)c.head_dim_qk));
    p->items.swap(items);
    p->num_tiles = ntiles;
    p->num_splits = nsplit;
    p->tokens = cu_q[num_segments];
    p->pairs = pairs;
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
    info->block_m = BM;
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

template <int DQK, int DV>
hipError_t launch(const AttnArgs& a, bool split, const CombineArgs& ca, hipStream_t stream) {
    const int64_t total = (int64_t)a.num_items * a.num_heads;
    if (total <= 0) return hipSuccess;
    if (total > (int64_t)INT32_MAX) return hipErrorInvalidValue;
    dim3 grid((unsigned)total), block(NTHREADS);
    if (split) {
        hipLaunchKernelGGL((attn_fwd_kernel<DQK, DV, true>), grid, block, 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t threads = (int64_t)ca.tokens * ca.num_heads * (DV / 4);
        dim3 cg((unsigned)((threads + 255) / 256));
        hipLaunchKernelGGL((combine_kernel<DV>), cg, dim3(256), 0, stream, ca);
    } else {
        hipLaunchKernelGGL((attn_fwd_kernel<DQK, DV, false>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

int env_xcd_remap() {
    const char* s = getenv("VPP_XCD_REMAP");
    return s ? atoi(s) : 1;
}

}  // namespace

extern "C" vpp_status_t vpp_chunk_attn_run(vpp_chunk_attn_plan_t p, const void* q, int64_t q_st, int64_t q_sh,
                                           const void* k, int64_t k_st, int64_t k_sh, const void* v,
                                           int64_t v_st, int64_t v_sh, void* out, int64_t o_st, int64_t o_sh,
                                           float* lse, int64_t lse_sh, void* workspace, size_t workspace_bytes,
                                           void* stream_ptr) {
    if (!p) return VPP_ERR_INVALID_ARG;
    if (!q || !k || !v || !out) return VPP_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return VPP_ERR_INVALID_ARG;
    if (!stride_ok(q_st) || !stride_ok(q_sh) || !stride_ok(k_st) || !stride_ok(k_sh) || !stride_ok(v_st) ||
        !stride_ok(v_sh) || !stride_ok(o_st) || !stride_ok(o_sh))
        return VPP_ERR_INVALID_ARG;
    if (lse && (((uintptr_t)lse & 3u) != 0 || lse_sh < p->tokens)) return VPP_ERR_INVALID_ARG;
    if (!workspace || ((uintptr_t)workspace & 255u) != 0) return VPP_ERR_WORKSPACE;
    if (workspace_bytes < p->ws_bytes) return VPP_ERR_WORKSPACE;
    if (p->items.empty()) return VPP_OK;  // nothing to do: every segment is empty

    hipStream_t stream = (hipStream_t)stream_ptr;
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
    char* ws = (char*)workspace;
    if (hipMemcpyAsync(ws, p->staging[slot], p->items_bytes, hipMemcpyHostToDevice, stream) != hipSuccess)
        return VPP_ERR_HIP;
    if (hipEventRecord(p->staging_done[slot], stream) != hipSuccess) return VPP_ERR_HIP;
    p->staging_pending[slot] = true;

    const vpp_chunk_attn_config_t& c = p->cfg;
    AttnArgs a;
    memset(&a, 0, sizeof a);
    a.items = (const WorkItem*)ws;
    a.q = (const u16*)q;
    a.k = (const u16*)k;
    a.v = (const u16*)v;
    a.out = (u16*)out;
    a.lse = lse;
    a.q_st = q_st; a.q_sh = q_sh; a.k_st = k_st; a.k_sh = k_sh; a.v_st = v_st; a.v_sh = v_sh;
    a.o_st = o_st; a.o_sh = o_sh; a.lse_sh = lse_sh;
    a.num_items = (int32_t)p->items.size();
    a.num_heads = c.num_q_heads;
    a.group = c.num_q_heads / c.num_kv_heads;
    a.tokens = p->tokens;
    a.scale_log2 = (float)((double)p->scale * 1.4426950408889634);
    a.xcd_remap = env_xcd_remap();
    const bool split = p->num_splits > 1;
    CombineArgs ca;
    memset(&ca, 0, sizeof ca);
    if (split) {
        size_t off = align256(p->items_bytes);
        a.part_o = (float*)(ws + off);
        off += align256((size_t)p->num_splits * p->tokens * c.num_q_heads * c.head_dim_v * sizeof(float));
        a.part_lse = (float*)(ws + off);
        ca.part_o = a.part_o;
        ca.part_lse = a.part_lse;
        ca.out = (u16*)out;
        ca.lse = lse;
        ca.o_st = o_st; ca.o_sh = o_sh; ca.lse_sh = lse_sh;
        ca.tokens = p->tokens;
        ca.num_heads = c.num_q_heads;
        ca.splits = p->num_splits;
    }
    hipError_t e;
    if (c.head_dim_qk == 64) e = launch<64, 64>(a, split, ca, stream);
    else if (c.head_dim_qk == 128) e = launch<128, 128>(a, split, ca, stream);
    else e = launch<192, 128>(a, split, ca, stream);
    return e == hipSuccess ? VPP_OK : VPP_ERR_HIP;
}

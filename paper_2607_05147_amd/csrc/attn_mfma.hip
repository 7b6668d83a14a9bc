// Ragged causal verify attention, bf16, head dim 128, on gfx950 matrix cores.
//
// Work item = (request r, KV head g, KV split s, row chunk rc).  The rows of a
// request are its q_len verify tokens times the GQA group, packed
// row = t * group + head_in_group.  A workgroup has four waves; the 16-row
// tiles of the chunk (64 * TPW rows) are dealt to them round-robin, and all
// four share the key/value stream of the split through LDS:
//
//   * the split (at most 4096 keys) is walked in 32-key steps; each step's
//     K and V rows (8 KB each) are copied from their page straight into LDS
//     with global_load_lds_dwordx4 (no registers involved), into a ring of
//     four buffers, three steps ahead of the one being computed; the waits
//     for those copies are explicit vmcnt counts;
//   * S^T[key, row] = K Q^T with v_mfma_f32_16x16x32_bf16: K fragments are
//     16-byte LDS reads (A operand), the wave's Q fragments stay in registers
//     (B operand); the key order inside a step is permuted so that the score
//     accumulator already has the B-operand layout of the next product;
//   * online softmax per row (exp2 of log2e-scaled scores, causal and length
//     masks), P rounded to bf16;
//   * O^T[d, row] += V^T P^T, V^T fragments read with ds_read_b64_tr_b16
//     (two transposing 8-byte reads per 16 x 32 fragment).
// LDS rows are 256 bytes; the 16-byte chunks of a row are XOR-swizzled (the
// copy chooses which chunk each lane fetches) so that the K fragment reads and
// the transposing V reads are free of bank conflicts.  Page ids of the split
// are loaded once (one per lane) and picked per step with readlane.
//
// The workgroups are persistent and take items from a list that a one-block
// plan kernel builds on the device, longest first.  A request whose context
// has more than one split stores per-split partials (m, l, unnormalised o);
// a merge kernel combines them afterwards in split order (bitwise
// reproducible).  Exchanging them across a kernel boundary needs no
// device-scope fences, which on this part would write back and invalidate the
// whole L2 of an XCD.
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace dspark {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMfThreads = 256;
constexpr int kMfWaves = 4;
// Keys per split (the last split of a context holds the rest): kSplit, or a
// smaller power of two down to kMinSplit when a batch's largest possible number
// of work items at kSplit is below kTargetItems (three rounds of the 512
// resident workgroups), so that a small batch still fills the part.
constexpr int kSplit = 4096;
constexpr int kMinSplit = 512;
constexpr int64_t kTargetItems = 1536;
static_assert(kSplit / 64 <= DSPARK_WAVE, "a split's page ids fit one per lane");
constexpr int kStepTok = 32;   // keys per step
constexpr int kRing = 4;       // LDS buffers; copies run kRing - 1 steps ahead
constexpr int kD = 128;
constexpr int kRowBytes = kD * 2;
constexpr int kTileBytes = kStepTok * kRowBytes;  // 8 KB
constexpr int kCopiesPerStep = 4;                 // 16-byte copies per thread per step
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Two 16-row tiles per wave when a request can have more than 64 rows.
static int pick_tpw(const AttnArgs& a) { return a.max_q * (a.Hq / a.Hkv) > 64 ? 2 : 1; }

bool attn_mfma_supported(const AttnArgs& a) {
    // power-of-two pages of 64 keys or more: a split (kSplit keys, aligned) then
    // spans at most 64 pages, whose ids fit one per lane of a wave
    const int64_t lim = (int64_t)1 << 30;  // byte strides fit 32-bit offsets
    return a.bf16 && a.Dqk == kD && a.Dv == kD && a.page >= 64 && (a.page & (a.page - 1)) == 0 &&
           a.ks[0] < lim && a.ks[1] < lim && a.ks[2] < lim && a.vs[0] < lim && a.vs[1] < lim &&
           a.vs[2] < lim && a.ks[2] > 0 && a.vs[2] > 0 &&
           a.Hq % a.Hkv == 0 && a.ks[2] % 8 == 0 && a.vs[2] % 8 == 0 && a.ks[1] % 8 == 0 &&
           a.vs[1] % 8 == 0 && a.ks[0] % 8 == 0 && a.vs[0] % 8 == 0 &&
           ((uintptr_t)a.q % 16) == 0 && ((uintptr_t)a.k % 16) == 0 &&
           ((uintptr_t)a.v % 16) == 0 && ((uintptr_t)a.out % 8) == 0;
}

struct MfGeom {
    int tpw, chunk_rows, group, split, max_splits, rc_max;
    int64_t n_items;   // upper bound on attention work items
    int64_t n_merge;   // upper bound on merge items (8 rows each)
    size_t counter_bytes, list_bytes, mlist_bytes, slot_floats, part_bytes;
};

constexpr int kMergeRows = 8;  // rows per merge item (32 threads of 4 values per row)

static MfGeom mf_geom(const AttnArgs& a) {
    MfGeom g;
    g.tpw = pick_tpw(a);
    g.chunk_rows = 16 * kMfWaves * g.tpw;
    g.group = a.Hq / a.Hkv;
    const int64_t max_kv = (int64_t)a.max_pages * a.page;
    g.rc_max = (a.max_q * g.group + g.chunk_rows - 1) / g.chunk_rows;
    const int64_t slots = (int64_t)a.R * a.Hkv * g.rc_max;
    g.split = kSplit;
    while (g.split > kMinSplit && slots * ((max_kv + g.split - 1) / g.split) < kTargetItems)
        g.split >>= 1;
    g.max_splits = (int)std::max<int64_t>(1, (max_kv + g.split - 1) / g.split);
    g.n_items = slots * g.max_splits;
    g.n_merge = g.max_splits > 1 ? slots * (g.chunk_rows / kMergeRows) : 0;
    // [0] next item, [1] number of items, [2] number of merge items
    g.counter_bytes = 256;
    g.list_bytes = ((size_t)g.n_items * 2 * sizeof(int4) + 255) & ~(size_t)255;
    g.mlist_bytes = ((size_t)g.n_merge * 2 * sizeof(int4) + 255) & ~(size_t)255;
    g.slot_floats = (size_t)g.chunk_rows * (kD + 2);
    g.part_bytes = g.max_splits > 1 ? (size_t)slots * g.max_splits * g.slot_floats * sizeof(float) : 0;
    return g;
}

size_t attn_mfma_workspace(const AttnArgs& a) {
    const MfGeom g = mf_geom(a);
    return g.counter_bytes + g.list_bytes + g.mlist_bytes + g.part_bytes;
}

struct MfParams {
    AttnArgs a;
    int group, split, max_splits, rc_max, chunk_rows;  // split: keys per split
    int page_shift;                      // log2(page size)
    uint32_t ks0b, ks1b, ks2b, vs0b, vs1b, vs2b;  // KV strides in bytes
    float scale2;
    int* work;      // [0] next item, [1] number of items, [2] number of merge items
    int4* list;     // attention items, two int4 each: {r, g, split, row chunk}, {q0, q_len, kv, splits}
    int4* mlist;    // merge items: {r, g, row chunk, first row in chunk}, {q0, q_len, kv, splits}
    float* part;    // split partials: [slot][split] {m[rows], l[rows], o[rows][128]}
};

// Keys [start, end) of split s of a context of kv keys: whole pieces of
// `split` keys, the last one holding the remainder.  The remainders spread item
// lengths down to a single step, so the longest-first list ends with short
// items and the persistent workgroups finish close together.
__host__ __device__ __forceinline__ void split_range(int kv, int split, int s, int& start, int& end) {
    start = s * split;
    end = min(kv, start + split);
}

// Builds the work lists on the device from cu_q / kv_len (no host round trip).
// One workgroup; eight threads per request (one per KV head, in turn).
// Attention items are placed longest first (a counting sort on their step
// count), so that the persistent workgroups end together; merge items list the
// 8-row groups of every (request, KV head, row chunk) that has more than one
// split.
constexpr int kPlanThreads = 1024;
constexpr int kPlanLanes = 8;                 // threads per request
constexpr int kBins = kSplit / kStepTok + 1;  // steps per item are at most kSplit / 32
constexpr int kBinsPerLane = (kBins + DSPARK_WAVE - 1) / DSPARK_WAVE;
__global__ __launch_bounds__(kPlanThreads) void mf_plan(MfParams p) {
    const AttnArgs& a = p.a;
    __shared__ int s_bin[kBins];
    __shared__ int s_merge;
    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int sub = tid % kPlanLanes;
    const int leader = lane & ~(kPlanLanes - 1);  // the request's first lane
    for (int i = tid; i < kBins; i += kPlanThreads) s_bin[i] = 0;
    if (tid == 0) s_merge = 0;
    __syncthreads();
    const int total_rows = min(max(a.cu_q[a.R], 0), a.R * a.max_q);
    auto shape = [&](int r, int& q0, int& ql, int& kv, int& ns, int& nr) {
        q0 = a.cu_q[r];
        ql = a.cu_q[r + 1] - q0;
        kv = a.kv_len[r];
        if (ql < 1 || ql > a.max_q || kv < ql || kv > a.max_pages * a.page) return false;
        // the request's rows must lie inside the flattened batch the caller
        // sized: [0, min(cu_q[R], R * max_q))
        if (q0 < 0 || (int64_t)q0 + ql > total_rows) return false;
        ns = (kv + p.split - 1) / p.split;
        nr = (ql * p.group + p.chunk_rows - 1) / p.chunk_rows;
        return true;
    };
    auto steps_of = [&](int kv, int ns, int sp) {
        int st, en;
        split_range(kv, p.split, sp, st, en);
        return min((en - st + kStepTok - 1) / kStepTok, kBins - 1);
    };
    // histogram of item lengths (the request's lanes share its splits)
    for (int r = tid / kPlanLanes; r < a.R; r += kPlanThreads / kPlanLanes) {
        int q0, ql, kv, ns, nr;
        if (!shape(r, q0, ql, kv, ns, nr)) continue;
        for (int sp = sub; sp < ns; sp += kPlanLanes) atomicAdd(&s_bin[steps_of(kv, ns, sp)], a.Hkv * nr);
    }
    __syncthreads();
    if (tid < DSPARK_WAVE) {
        // bin start offsets, longest first: lane l owns the bins at descending
        // positions kBinsPerLane * l .. kBinsPerLane * (l + 1) - 1
        int cnt[kBinsPerLane], mine = 0;
#pragma unroll
        for (int k = 0; k < kBinsPerLane; ++k) {
            const int b = kBins - 1 - (kBinsPerLane * lane + k);
            cnt[k] = b >= 0 ? s_bin[b] : 0;
            mine += cnt[k];
        }
        int incl = mine;
        for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
            const int t = __shfl_up(incl, o, DSPARK_WAVE);
            if (lane >= o) incl += t;
        }
        int run = incl - mine;
#pragma unroll
        for (int k = 0; k < kBinsPerLane; ++k) {
            const int b = kBins - 1 - (kBinsPerLane * lane + k);
            if (b >= 0) s_bin[b] = run;
            run += cnt[k];
        }
        if (lane == DSPARK_WAVE - 1) {
            p.work[0] = 0;
            p.work[1] = incl;
        }
    }
    __syncthreads();
    for (int r = tid / kPlanLanes; r < a.R; r += kPlanThreads / kPlanLanes) {
        int q0, ql, kv, ns, nr;
        if (!shape(r, q0, ql, kv, ns, nr)) continue;  // the same for the request's lanes
        const int4 meta = int4{q0, ql, kv, ns};
        for (int sp = 0; sp < ns; ++sp) {
            // the KV heads and row chunks of one split stay next to each other
            int base = 0;
            if (sub == 0) base = atomicAdd(&s_bin[steps_of(kv, ns, sp)], a.Hkv * nr);
            base = __shfl(base, leader, DSPARK_WAVE);
            for (int g = sub; g < a.Hkv; g += kPlanLanes)
                for (int rc = 0; rc < nr; ++rc) {
                    const int off = base + g * nr + rc;
                    p.list[2 * off] = int4{r, g, sp, rc};
                    p.list[2 * off + 1] = meta;
                }
        }
        if (ns > 1) {
            const int rows = ql * p.group;
            int cnt = 0;  // merge groups per KV head
            for (int rc = 0; rc < nr; ++rc)
                cnt += (min(p.chunk_rows, rows - rc * p.chunk_rows) + kMergeRows - 1) / kMergeRows;
            int base = 0;
            if (sub == 0) base = atomicAdd(&s_merge, a.Hkv * cnt);
            base = __shfl(base, leader, DSPARK_WAVE);
            for (int g = sub; g < a.Hkv; g += kPlanLanes) {
                int off = base + g * cnt;
                for (int rc = 0; rc < nr; ++rc) {
                    const int nrows = min(p.chunk_rows, rows - rc * p.chunk_rows);
                    for (int m0 = 0; m0 < nrows; m0 += kMergeRows, ++off) {
                        p.mlist[2 * off] = int4{r, g, rc, m0};
                        p.mlist[2 * off + 1] = meta;
                    }
                }
            }
        }
    }
    __syncthreads();
    if (tid == 0) p.work[2] = s_merge;
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// 16-byte chunk slot of chunk c in LDS row t (t < 32) of the K / V tile.  gfx950
// serves a 16-byte LDS read in four 16-lane phases (lanes split by bit 5 and
// by the parity of bits 2 ^ 3 ^ 4) and a transposing 8-byte read in two
// 32-lane halves, over 64 four-byte banks; with 256-byte rows these XORs put
// every phase of the score-operand reads (k_slot) and of the value-operand
// reads (v_slot) on distinct banks.  Both maps are involutions on 0..15.
__device__ __forceinline__ int k_slot(int t, int c) { return c ^ ((t & 3) | (((t >> 3) & 3) << 2)); }
__device__ __forceinline__ int v_slot(int t, int c) { return c ^ (((t & 3) | (((t >> 3) & 1) << 2)) << 1); }

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

// A head-dim row of zeros in device memory (zero-initialised at load, never
// written): keys at or past a split's end are copied from here instead of
// from the page, so stale or NaN page tails never reach LDS.
__device__ __align__(16) uint16_t g_zero_row[kD];

// 16-byte copy global -> LDS for a whole wave: lane L's 16 bytes land at
// lds_base + 16 L (lds_base is wave-uniform).  Emitted as inline asm so that
// the compiler does not add its own conservative waits for it; the kernel
// waits for these copies with explicit vmcnt counts.
__device__ __forceinline__ void lds_copy16(const void* gsrc, uint32_t lds_addr) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(m0), "v"(gsrc)
        : "memory", "m0");
}

// s_waitcnt vmcnt(N) leaving the other counters alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// NaN-propagating maximum (v_maximum3_f32; no operand canonicalisation)
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// max over the four lanes that share a row (lanes lr, lr + 16, lr + 32, lr + 48)
__device__ __forceinline__ float row_max4(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

// copy with a wave-uniform 64-bit base (SGPRs) and a per-lane 32-bit offset
__device__ __forceinline__ void lds_copy16_s(uint64_t sbase, uint32_t voff, uint32_t lds_addr) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_addr);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)sbase);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(sbase >> 32));
    const uint64_t sb = ((uint64_t)hi << 32) | lo;
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "global_load_lds_dwordx4 %1, %2"
        :
        : "s"(m0), "v"(voff), "s"(sb)
        : "memory", "m0");
}

constexpr float kRescale = 8.0f;  // log2 headroom before the running max is moved

template <int TPW>
__device__ __forceinline__ void attn_item(const MfParams& p, const int r, const int g, const int s,
                                          const int rc, const int q0, const int ql, const int kv,
                                          const int nsplit, const uint32_t lds0, int& nxt) {
    const AttnArgs& a = p.a;
    constexpr int kChunkRows = 16 * kMfWaves * TPW;
    constexpr int kSlotFloats = kChunkRows * (kD + 2);
    const int rg = r * a.Hkv + g;
    // the plan only lists valid items: 1 <= ql <= max_q, ql <= kv <= max_pages * page,
    // s < nsplit, rc * kChunkRows < ql * group
    const int rows = ql * p.group;
    const int row0 = rc * kChunkRows;
    int start, end;
    split_range(kv, p.split, s, start, end);
    const int nrows = min(kChunkRows, rows - row0);
    const int nt = (nrows + 15) >> 4;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int lr = lane & 15;
    const int lq = lane >> 4;
    // tiles are dealt round-robin: wave w owns tiles w, w + 4, ...
    const int nt_w = nt > wave ? min((nt - wave + kMfWaves - 1) / kMfWaves, TPW) : 0;

    const uint16_t* __restrict__ qg = (const uint16_t*)a.q;
    const uint16_t* __restrict__ kc = (const uint16_t*)a.k;
    const uint16_t* __restrict__ vc = (const uint16_t*)a.v;

    // ---- page ids of the split, one per lane
    const int pg0 = start >> p.page_shift;
    const int npg = ((end - 1) >> p.page_shift) - pg0 + 1;  // <= 64 (pages of >= 64 keys)
    const int my_page = lane < npg ? a.block_table[(int64_t)r * a.max_pages + pg0 + lane] : 0;

    // ---- query fragments (B operand of S^T = K Q^T) and causal limits
    bf16x8 qf[TPW][4];
    int lim[TPW];
    int lim_min = 0x7fffffff;  // smallest causal limit of this wave's rows
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int row = row0 + 16 * (wave + kMfWaves * j) + lr;
        if (row < rows) {
            const int t = row / p.group;
            const int h = g * p.group + (row - t * p.group);
            const uint16_t* qp = qg + ((int64_t)(q0 + t) * a.Hq + h) * kD + 8 * lq;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) qf[j][ks] = *(const bf16x8*)(qp + 32 * ks);
            lim[j] = kv - ql + t;
            if (j < nt_w) lim_min = min(lim_min, lim[j]);
        } else {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) qf[j][ks] = bf16x8{};
            lim[j] = -1;
        }
    }
    lim_min = __reduce_min_sync(~0ull, lim_min);

    f32x4 acc[TPW][8];
    float mrow[TPW], lsum[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        mrow[j] = -__builtin_huge_valf();
        lsum[j] = 0.0f;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[j][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // ---- per-lane LDS offsets of the MFMA fragments (loop invariant)
    int koff[2][4];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const int t = 8 * (lr >> 2) + 4 * mb + (lr & 3);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            koff[mb][ks] = lds0 + t * kRowBytes + k_slot(t, 4 * ks + lq) * 16;
    }
    int voff[8][2];
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int t = 8 * lq + 4 * h + (lr >> 2);
            const int c = 2 * db + ((lr & 3) >> 1);
            voff[db][h] = lds0 + kTileBytes + t * kRowBytes + v_slot(t, c) * 16 + (lr & 1) * 8;
        }

    // ---- copy geometry: wave w, copy i (0, 1) fills LDS slots (2w + i) * 64 + lane
    // of a 512-slot tile: row t = 4 (2w + i) + lane / 16, physical chunk lane % 16,
    // which holds source chunk (physical ^ swizzle(t)).
    int cp_row[2], cp_kchunk[2], cp_vchunk[2];
    uint32_t cp_koff[2], cp_voff[2];  // byte offsets from the step's first key
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int t = 4 * (2 * wave + i) + (lane >> 4);
        cp_row[i] = t;
        cp_kchunk[i] = k_slot(t, lane & 15);  // the map is an involution
        cp_vchunk[i] = v_slot(t, lane & 15);
        cp_koff[i] = t * p.ks2b + 16 * cp_kchunk[i];
        cp_voff[i] = t * p.vs2b + 16 * cp_vchunk[i];
    }
    const int nsteps = (end - start + kStepTok - 1) / kStepTok;  // >= 1
    const int last = nsteps - 1;
    // this wave's copy destinations start 2 KB into each tile (wave-uniform)
    const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds0 + wave * 2048);
    const uint64_t kc_head = (uint64_t)(uintptr_t)kc + (uint64_t)((uint32_t)g * p.ks1b);
    const uint64_t vc_head = (uint64_t)(uintptr_t)vc + (uint64_t)((uint32_t)g * p.vs1b);

    auto issue = [&](int n) {
        const int tok0 = start + n * kStepTok;
        const int page = __builtin_amdgcn_readlane(my_page, (tok0 >> p.page_shift) - pg0);
        const int slot0 = tok0 & ((1 << p.page_shift) - 1);
        const uint32_t kd = lds_wave + ((unsigned)n & (kRing - 1)) * (2 * kTileBytes);
        const uint32_t vd = kd + kTileBytes;
        if (tok0 + kStepTok <= end) {
            const uint64_t kb = kc_head + (uint64_t)(uint32_t)page * p.ks0b + (uint32_t)slot0 * p.ks2b;
            const uint64_t vb = vc_head + (uint64_t)(uint32_t)page * p.vs0b + (uint32_t)slot0 * p.vs2b;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                lds_copy16_s(kb, cp_koff[i], kd + i * 1024);
                lds_copy16_s(vb, cp_voff[i], vd + i * 1024);
            }
        } else {
            // last, partial step: keys at or past the end come from the zero row
            const uint16_t* kb = kc + (int64_t)page * a.ks[0] + (int64_t)g * a.ks[1];
            const uint16_t* vb = vc + (int64_t)page * a.vs[0] + (int64_t)g * a.vs[1];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int64_t tr = slot0 + cp_row[i];
                const bool in = tok0 + cp_row[i] < end;
                const uint16_t* ksrc = in ? kb + tr * a.ks[2] + 8 * cp_kchunk[i] : g_zero_row + 8 * cp_kchunk[i];
                const uint16_t* vsrc = in ? vb + tr * a.vs[2] + 8 * cp_vchunk[i] : g_zero_row + 8 * cp_vchunk[i];
                lds_copy16(ksrc, kd + i * 1024);
                lds_copy16(vsrc, vd + i * 1024);
            }
        }
    };

    auto compute = [&](int n, auto bufc) {
        constexpr unsigned buf = decltype(bufc)::value;
        const int tok0 = start + n * kStepTok;
        constexpr uint32_t boff = buf * (2 * kTileBytes);
        // all K fragments of the step first (8 LDS reads in flight), then the scores
        bf16x8 kfr[2][4];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) kfr[mb][ks] = *lds_ptr<const lds_bf16x8>(koff[mb][ks] + boff);
        f32x4 sc[TPW][2];
#pragma unroll
        for (int j = 0; j < TPW; ++j)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                sc[j][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (j < nt_w)
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks)
                        sc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kfr[mb][ks], qf[j][ks], sc[j][mb], 0, 0, 0);
            }
        // V^T fragments (16 transposing reads in flight) while the softmax runs.
        bf16x8 vfr[8];
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const s16x4 h0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                lds_ptr<lds_s16x4>(voff[db][0] + boff));
            const s16x4 h1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                lds_ptr<lds_s16x4>(voff[db][1] + boff));
            vfr[db] = __builtin_bit_cast(
                bf16x8, (short __attribute__((ext_vector_type(8)))){h0[0], h0[1], h0[2], h0[3],
                                                                     h1[0], h1[1], h1[2], h1[3]});
        }
        // keys of this lane: tok0 + 8 lq + 4 mb + e; masks only where needed
        const bool full = tok0 + kStepTok <= end && tok0 + kStepTok - 1 <= lim_min;
        bf16x8 pf[TPW];
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            if (j < nt_w) {
                // raw scores; the scale is applied inside the exponent below
                float sv[8];
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) sv[4 * mb + e] = sc[j][mb][e];
                if (!full) {
#pragma unroll
                    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int key = tok0 + 8 * lq + 4 * mb + e;
                            if (!(key < end && key <= lim[j])) sv[4 * mb + e] = -__builtin_huge_valf();
                        }
                }
                float bm = vmax(vmax(vmax(sv[0], sv[1]), sv[2]),
                                vmax(vmax(sv[3], sv[4]), vmax(vmax(sv[5], sv[6]), sv[7])));
                bm = row_max4(bm) * p.scale2;
                // move the running max only when the new one exceeds it by kRescale
                // (P stays below 2^kRescale; the result is normalised at the end)
                const bool need = bm > mrow[j] + kRescale;
                if (__builtin_amdgcn_ballot_w64(need)) {
                    const float mn = need ? bm : mrow[j];
                    const float alpha = need ? __builtin_amdgcn_exp2f(mrow[j] - mn) : 1.0f;
                    lsum[j] *= alpha;
#pragma unroll
                    for (int db = 0; db < 8; ++db) acc[j][db] *= alpha;
                    mrow[j] = mn;
                }
                const float mu = mrow[j] == -__builtin_huge_valf() ? 0.0f : mrow[j];
                float pr[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) pr[k] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[k], p.scale2, -mu));
                lsum[j] += ((pr[0] + pr[1]) + (pr[2] + pr[3])) + ((pr[4] + pr[5]) + (pr[6] + pr[7]));
                // k-slot 8 lq + i <-> key 8 lq + i: M-block 0 gives i = 0..3, M-block 1 i = 4..7
                u32x4 pk;
                pk[0] = cvt_pk_bf16(pr[0], pr[1]);
                pk[1] = cvt_pk_bf16(pr[2], pr[3]);
                pk[2] = cvt_pk_bf16(pr[4], pr[5]);
                pk[3] = cvt_pk_bf16(pr[6], pr[7]);
                pf[j] = __builtin_bit_cast(bf16x8, pk);
            }
        }
#pragma unroll
        for (int j = 0; j < TPW; ++j)
            if (j < nt_w)
#pragma unroll
                for (int db = 0; db < 8; ++db)
                    acc[j][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vfr[db], pf[j], acc[j][db], 0, 0, 0);
    };

    // ---- main loop.  Every thread issues kCopiesPerStep copies per step, in step
    // order, also past the last step (copies of the zero row into buffers that
    // are not read again), so "step n has landed" is always
    // vmcnt <= (kRing - 2) * kCopiesPerStep.  Keys past the split end are copied
    // as zeros (masked scores, zero values).  The loop is unrolled by the ring
    // size so that every LDS address is a per-lane base plus an immediate.
    wait_vmcnt<0>();
#pragma unroll
    for (int n = 0; n < kRing - 1; ++n) issue(n);
    // the next item is claimed three steps before this one ends: late enough
    // that no claimed item waits behind a long one, early enough for the
    // atomic to return before the end (it adds one operation to wave 0's
    // count, which at worst makes one wait cover a copy of the next step too)
    const int claim = max(nsteps - 3, 0);
    auto one = [&](int n, auto bufc) {
        wait_vmcnt<(kRing - 2) * kCopiesPerStep>();
        lds_barrier();  // step n visible to all; everyone is done with step n - 1
        if (n == claim && tid == 0) nxt = atomicAdd(p.work, 1);
        issue(n + kRing - 1);
        if (nt_w > 0) compute(n, bufc);
    };
    for (int n = 0; n < nsteps; n += kRing) {
        one(n, std::integral_constant<unsigned, 0>{});
        if (n + 1 < nsteps) one(n + 1, std::integral_constant<unsigned, 1>{});
        if (n + 2 < nsteps) one(n + 2, std::integral_constant<unsigned, 2>{});
        if (n + 3 < nsteps) one(n + 3, std::integral_constant<unsigned, 3>{});
    }
    wait_vmcnt<0>();

    // ---- finish rows: total l over the four lanes of a row
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        lsum[j] += __shfl_xor(lsum[j], 16, 64);
        lsum[j] += __shfl_xor(lsum[j], 32, 64);
    }
    uint16_t* outp = (uint16_t*)a.out;
    if (nsplit == 1) {
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int row = row0 + 16 * (wave + kMfWaves * j) + lr;
            if (j < nt_w && row < rows) {
                const int t = row / p.group;
                const int h = g * p.group + (row - t * p.group);
                const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
                const float inv = 1.0f / lsum[j];
#pragma unroll
                for (int db = 0; db < 8; ++db) {
                    uint2 pk;
                    pk.x = pack2_bf16(acc[j][db][0] * inv, acc[j][db][1] * inv);
                    pk.y = pack2_bf16(acc[j][db][2] * inv, acc[j][db][3] * inv);
                    *(uint2*)(outp + orow * kD + 16 * db + 4 * lq) = pk;
                }
                if (a.lse && lq == 0) a.lse[orow] = (mrow[j] + log2f(lsum[j])) * kLn2;
            }
        }
        return;
    }

    // ---- several splits: store this split's partial (m, l, unnormalised o);
    // the merge kernel combines them after this kernel has ended
    float* part = p.part + (((int64_t)rg * p.rc_max + rc) * p.max_splits + s) * kSlotFloats;
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
        const int rr = 16 * (wave + kMfWaves * j) + lr;
        if (j < nt_w) {
            if (lq == 0) {
                part[rr] = mrow[j];
                part[kChunkRows + rr] = lsum[j];
            }
#pragma unroll
            for (int db = 0; db < 8; ++db)
                *(f32x4*)(part + 2 * kChunkRows + rr * kD + 16 * db + 4 * lq) = acc[j][db];
        }
    }
}

// Persistent workgroups pull items from the device-built list.
template <int TPW>
__global__ __launch_bounds__(kMfThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_mfma_kernel(MfParams p) {
    __shared__ __align__(16) unsigned char lds[kRing][2][kTileBytes];  // [buffer][K | V]
    __shared__ int s_item;
    // the ring's LDS address as a plain integer (all LDS addressing below is
    // integer arithmetic on it)
    uint32_t lds0 = (uint32_t)(uintptr_t)&lds[0][0][0];
    asm volatile("" : "+s"(lds0));
    const int total = p.work[1];
    if (threadIdx.x == 0) s_item = atomicAdd(p.work, 1);
    __syncthreads();
    int it = __builtin_amdgcn_readfirstlane(s_item);
    while (it < total) {
        const int4 e0 = p.list[2 * it];      // uniform: scalar loads
        const int4 e1 = p.list[2 * it + 1];
        int nxt = 0;  // claimed by thread 0 near the end of the item
        attn_item<TPW>(p, e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w, lds0, nxt);
        __syncthreads();  // everyone is done with this item's LDS and s_item
        if (threadIdx.x == 0) s_item = nxt;
        __syncthreads();
        it = __builtin_amdgcn_readfirstlane(s_item);
    }
}

// Combines the split partials of one 8-row group: 32 threads per row, four
// values each.  The partials of up to kMergeBatch splits are loaded in one
// round (o does not depend on the row max), then combined in split order
// (bitwise reproducible).
constexpr int kMergeBatch = 8;
template <int TPW>
__global__ __launch_bounds__(256) void attn_mfma_merge(MfParams p) {
    constexpr int kChunkRows = 16 * kMfWaves * TPW;
    constexpr int kSlotFloats = kChunkRows * (kD + 2);
    const AttnArgs& a = p.a;
    const int count = p.work[2];
    const int tid = threadIdx.x;
    // the first item's entries are loaded together with the count: the list
    // has room for at least gridDim.x items (the launch caps the grid at its
    // capacity), and entries past the count are never used
    int4 e0 = p.mlist[2 * blockIdx.x];
    int4 e1 = p.mlist[2 * blockIdx.x + 1];
    for (int m = blockIdx.x; m < count; m += gridDim.x) {
        if (m != (int)blockIdx.x) {
            e0 = p.mlist[2 * m];
            e1 = p.mlist[2 * m + 1];
        }
        const int r = e0.x, g = e0.y, rc = e0.z;
        const int q0 = e1.x, ql = e1.y, ns = e1.w;
        const int rows = ql * p.group;
        const int nrows = min(kChunkRows, rows - rc * kChunkRows);
        const int mr = e0.w + (tid >> 5);  // row inside the chunk
        if (mr >= nrows) continue;
        const int c4 = (tid & 31) * 4;
        const float* base = p.part + ((int64_t)(r * a.Hkv + g) * p.rc_max + rc) * p.max_splits * kSlotFloats;
        float M = -__builtin_huge_valf();
        float L = 0.0f;
        f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int s0 = 0; s0 < ns; s0 += kMergeBatch) {
            float ms[kMergeBatch], ls[kMergeBatch];
            f32x4 os[kMergeBatch];
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const float* sl = base + (int64_t)min(s0 + k, ns - 1) * kSlotFloats;
                ms[k] = sl[mr];
                ls[k] = sl[kChunkRows + mr];
                os[k] = *(const f32x4*)(sl + 2 * kChunkRows + mr * kD + c4);
            }
            float Mb = M;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k)
                if (s0 + k < ns) Mb = fmaxf(Mb, ms[k]);
            // rescale what earlier batches accumulated (one batch when ns <= 8)
            if (M > -__builtin_huge_valf() && Mb != M) {
                const float f = exp2f(M - Mb);
                L *= f;
                o *= f;
            }
            M = Mb;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                if (s0 + k >= ns) break;
                const float f = ms[k] > -__builtin_huge_valf() ? exp2f(ms[k] - M) : 0.0f;
                L += ls[k] * f;
                o += f * os[k];
            }
        }
        const int row = rc * kChunkRows + mr;
        const int t = row / p.group;
        const int h = g * p.group + (row - t * p.group);
        const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
        const float inv = 1.0f / L;
        uint2 pk;
        pk.x = pack2_bf16(o[0] * inv, o[1] * inv);
        pk.y = pack2_bf16(o[2] * inv, o[3] * inv);
        *(uint2*)((uint16_t*)a.out + orow * kD + c4) = pk;
        if (a.lse && c4 == 0) a.lse[orow] = (M + log2f(L)) * kLn2;
    }
}

hipError_t launch_attn_mfma(const AttnArgs& a, void* ws, hipStream_t s) {
    const MfGeom g = mf_geom(a);
    MfParams p;
    p.a = a;
    p.group = g.group;
    p.split = g.split;
    p.max_splits = g.max_splits;
    p.rc_max = g.rc_max;
    p.chunk_rows = g.chunk_rows;
    p.scale2 = a.scale * kLog2e;
    p.page_shift = __builtin_ctz((unsigned)a.page);
    p.ks0b = (uint32_t)(a.ks[0] * 2);
    p.ks1b = (uint32_t)(a.ks[1] * 2);
    p.ks2b = (uint32_t)(a.ks[2] * 2);
    p.vs0b = (uint32_t)(a.vs[0] * 2);
    p.vs1b = (uint32_t)(a.vs[1] * 2);
    p.vs2b = (uint32_t)(a.vs[2] * 2);
    p.work = (int*)ws;
    p.list = (int4*)((char*)ws + g.counter_bytes);
    p.mlist = (int4*)((char*)ws + g.counter_bytes + g.list_bytes);
    p.part = (float*)((char*)ws + g.counter_bytes + g.list_bytes + g.mlist_bytes);
    hipLaunchKernelGGL(mf_plan, dim3(1), dim3(kPlanThreads), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // two resident workgroups per CU (64 KB of LDS and <= 256 VGPRs each)
    const int64_t grid = std::min<int64_t>((int64_t)cus * 2, std::max<int64_t>(g.n_items, 1));
    if (g.tpw == 2)
        hipLaunchKernelGGL(attn_mfma_kernel<2>, dim3((unsigned)grid), dim3(kMfThreads), 0, s, p);
    else
        hipLaunchKernelGGL(attn_mfma_kernel<1>, dim3((unsigned)grid), dim3(kMfThreads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess || g.n_merge == 0) return e;
    const int64_t mgrid = std::min<int64_t>((int64_t)cus * 16, g.n_merge);
    if (g.tpw == 2)
        hipLaunchKernelGGL(attn_mfma_merge<2>, dim3((unsigned)mgrid), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(attn_mfma_merge<1>, dim3((unsigned)mgrid), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace dspark

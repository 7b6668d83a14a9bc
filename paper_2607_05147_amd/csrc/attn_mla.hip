// Latent (MLA-style) verify attention on gfx950 matrix cores.
//
// Shape: query heads sharing one latent KV head per group, Dqk = 576 (512
// latent + 64 rotary dims), Dv = 512 with the values being the first 512 dims
// of the same cache rows, bf16.  With 128 query heads on one latent head every
// verify token contributes 128 rows that read the same keys, so the work is a
// dense contraction (about 1.2 kFLOP per KV byte): this path is MFMA-bound,
// unlike the GQA path.
//
// Work item = (request r, KV head g, block of 64 rows, KV split s).  A
// workgroup of eight waves owns the block, two per SIMD, in two roles:
//   * score waves (0-3) hold the query fragments of 32 rows each in
//     registers and compute S^T = K Q^T for one 16-key block of every step
//     with v_mfma_f32_16x16x32_bf16 (18 slices of the 576 dims), then the
//     softmax in exp2 units against a fixed per-row reference (the first
//     step's maximum; a block whose scores outgrow it by more than 2^32 runs
//     again with the observed maxima; masks only at the diagonal) and the bf16
//     probabilities, which go to the value waves through LDS;
//   * value waves (4-7) own 128 output dims of all 64 rows in the
//     accumulation registers, issue the step copies and compute
//     O^T += V^T P^T with the values read by ds_read_b64_tr_b16.
// Stage t runs the score waves on step t and the value waves on step t - 1,
// so each SIMD holds one wave of each role: one wave's softmax and operand
// waits run while the other's products keep the matrix core busy.  One LDS
// barrier ends a stage.  The split is walked in 32-key steps; each step's 32
// cache rows (36 KB) are copied into LDS with global_load_lds_dwordx4 (nine
// instructions per value wave) into a ring of four buffers, two steps ahead
// (a step is read by the score waves in stage t and by the value waves in
// stage t + 1).  LDS rows keep the 1152-byte cache pitch and the 16-byte
// chunks are swizzled (bits 0-2 of the chunk index XOR a function of the row,
// see pchunk) so that the score operand reads and the transposing value reads
// are free of bank conflicts while every read address stays a per-lane base
// plus an immediate.
// The row blocks of one (request, split) read the same keys: work items go to
// eight queues, one per XCD (workgroup b runs on XCD b % 8), so those blocks
// run side by side on one XCD and share its L2.  A workgroup whose queue is
// empty takes items from the others.  Splits of one row block are combined by
// a merge kernel after this one, in split order (bitwise reproducible).
#include <algorithm>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace dspark {
namespace mla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kDk = 576;
constexpr int kDv = 512;
constexpr int kThreads = 512;                       // 4 score waves + 4 value waves, two per SIMD
constexpr int kSW = 4;                              // score waves 0..3, value waves 4..7
constexpr int kVW = 4;
constexpr int kRows = 64;                           // rows per work item: four 16-row tiles
constexpr int kTilesPV = kRows / 16;                // tiles of the value product (all, per wave)
constexpr int kSTiles = 2;                          // tiles of the score product per wave
constexpr int kStep = 32;                           // keys per step
constexpr int kRing = 4;                            // step n sits in buffer n % 4; copies run 2 steps ahead
constexpr int kChunks = kDk / 8;                    // 72 16-byte chunks of a cache row
constexpr int kRowChunks = kChunks;                 // LDS row pitch in chunks (no pad: the swizzle spreads banks)
constexpr int kRowB = kRowChunks * 16;              // 1152 bytes
constexpr int kTileChunks = kStep * kRowChunks;     // 2304
constexpr int kTileB = kTileChunks * 16;            // 36864 bytes
constexpr int kInstr = kTileChunks / 64;            // 36 wave copy instructions per step
constexpr int kCopies = kInstr / kVW;               // 9 per value wave: 8 whole rows
constexpr int kSplit = 8192;                        // keys per split (the last one holds the rest)
constexpr int kPageRegs = (kSplit / 64 + DSPARK_WAVE - 1) / DSPARK_WAVE;  // page-id registers per lane (pages >= 64 keys)
constexpr int kKs = kDk / 32;                       // 18 slices of the score product
constexpr int kDb = kDv / 16;                       // 32 blocks of output dims
constexpr int kDbW = kDb / kVW;                     // 8 blocks (128 dims) per value wave
constexpr int kQueues = 8;                          // one per XCD
constexpr int kBins = kSplit / kStep + 1;           // item lengths in steps: 0 .. kSplit / 32
constexpr int kMergeRows = 4;                       // rows per merge item (64 threads per row)
constexpr int kAheadK = 6;                          // K fragment reads in flight ahead of the products
constexpr int kAheadV = 8;                          // transposing V reads in flight ahead of the products
constexpr int kSchedMfma = 0x008;                   // sched_group_barrier classes
constexpr int kSchedDsRead = 0x100;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRange = 32.0f;  // scores may exceed a row's reference by this (log2 units)
static_assert(kInstr == kVW * kCopies && kCopies * 64 == 8 * kRowChunks, "copy split over the value waves");
static_assert(kChunks % 8 == 0, "the swizzle permutes chunks within aligned groups of 8");
static_assert(kPageRegs * DSPARK_WAVE * 64 >= kSplit, "page ids of a split fit the lanes");

struct Geom {
    int group, rb_max, max_splits;
    int64_t n_items, n_merge;
    size_t head_bytes, list_bytes, mlist_bytes, slot_floats, part_bytes;
};

struct Params {
    AttnArgs a;
    int group, rb_max, max_splits, page_shift;
    uint32_t s0b, s1b, s2b;  // cache strides in bytes (values alias the keys)
    float scale2;
    int* head;               // [0..7] queue cursors, [8..15] queue begin, [16..23] queue end, [24] merges
    int4* list;              // items: {r, g, row block, split}, {q0, q_len, kv, splits}
    int4* mlist;             // merge items: {r, g, row block, first row}, {q0, q_len, kv, splits}
    float* part;             // [slot][split] {m[kRows], l[kRows], o[kRows][512]}
};

static Geom geom(const AttnArgs& a) {
    Geom g;
    g.group = a.Hq / a.Hkv;
    g.rb_max = (a.max_q * g.group + kRows - 1) / kRows;
    const int64_t max_kv = (int64_t)a.max_pages * a.page;
    g.max_splits = (int)std::max<int64_t>(1, (max_kv + kSplit - 1) / kSplit);
    const int64_t slots = (int64_t)a.R * a.Hkv * g.rb_max;
    g.n_items = slots * g.max_splits;
    g.n_merge = g.max_splits > 1 ? slots * (kRows / kMergeRows) : 0;
    g.head_bytes = 256;
    g.list_bytes = ((size_t)g.n_items * 2 * sizeof(int4) + 255) & ~(size_t)255;
    g.mlist_bytes = ((size_t)g.n_merge * 2 * sizeof(int4) + 255) & ~(size_t)255;
    g.slot_floats = (size_t)kRows * (kDv + 2);
    g.part_bytes = g.max_splits > 1 ? (size_t)slots * g.max_splits * g.slot_floats * sizeof(float) : 0;
    return g;
}

__host__ __device__ __forceinline__ void split_range(int kv, int s, int& start, int& end) {
    start = s * kSplit;
    end = min(kv, start + kSplit);
}

// Physical chunk of chunk c in LDS row t: bits 0-2 of c XOR (t % 4 | (t / 8 % 2) << 2).
// gfx950 serves a 16-byte LDS read in four 16-lane phases (lanes split by bit 5
// and by the parity of bits 2 ^ 3 ^ 4) and a transposing 8-byte read in two
// 32-lane halves, over 64 four-byte banks; with a 1152-byte pitch this XOR
// puts the 16 (or 32) lanes of every phase of the score-operand and the
// value-operand reads below on distinct banks.
__device__ __forceinline__ int pchunk(int t, int c) { return c ^ ((t & 3) | (((t >> 3) & 1) << 2)); }

// A cache row of zeros (zero-initialised at load, never written): keys at or
// past a split's end are copied from here.
__device__ __align__(16) uint16_t g_zero_row[kDk];

__device__ __forceinline__ void lds_copy16(const void* gsrc, uint32_t lds_addr) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(m0), "v"(gsrc)
        : "memory", "m0");
}

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

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

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

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// ------------------------------------------------------------------ plan

// Builds the per-XCD work queues and the merge list from cu_q / kv_len.  One
// workgroup.  Groups (request, KV head, split) are dealt to the queues round
// robin in request order; inside a queue the items are counting-sorted by
// length, longest first, with the row blocks of a group kept together.
// Every loop is spread over (request, split) or (request, merge item) pairs,
// so no thread runs a long chain of dependent LDS operations.
constexpr int kPlanThreads = 1024;
constexpr int kPlanMaxR = 8192;                                  // the ABI's limit on R
constexpr int kBinsPerLane = (kBins + DSPARK_WAVE - 1) / DSPARK_WAVE;
constexpr int kMergePerBlock = kRows / kMergeRows;               // merge items of a full row block
static_assert(kQueues <= kPlanThreads / DSPARK_WAVE, "one wave per queue");
__global__ __launch_bounds__(kPlanThreads) void mla_plan(Params p) {
    const AttnArgs& a = p.a;
    __shared__ int s_bin[kQueues][kBins];
    __shared__ int s_qstart[kQueues];
    __shared__ int s_wave[2][kPlanThreads / DSPARK_WAVE];
    __shared__ int s_gid0[kPlanMaxR];  // first group id of each request
    __shared__ int s_mb0[kPlanMaxR];   // first merge item of each request
    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    for (int i = tid; i < kQueues * kBins; i += kPlanThreads) (&s_bin[0][0])[i] = 0;
    const int total_rows = min(max(a.cu_q[a.R], 0), a.R * a.max_q);
    auto shape = [&](int r, int& q0, int& ql, int& kv, int& ns, int& nrb) {
        q0 = a.cu_q[r];
        ql = a.cu_q[r + 1] - q0;
        kv = a.kv_len[r];
        if (ql < 1 || ql > a.max_q || kv < ql || kv > a.max_pages * a.page) return false;
        // the request's rows must lie inside the flattened batch the caller
        // sized: [0, min(cu_q[R], R * max_q))
        if (q0 < 0 || (int64_t)q0 + ql > total_rows) return false;
        ns = (kv + kSplit - 1) / kSplit;
        nrb = (ql * p.group + kRows - 1) / kRows;
        return true;
    };
    auto steps_of = [&](int kv, int s) {
        int st, en;
        split_range(kv, s, st, en);
        return min((en - st + kStep - 1) / kStep, kBins - 1);
    };
    // merge items of one KV head of a request: 16 per full row block, the last block's rows / 4
    auto merges_of = [&](int ql, int ns, int nrb) {
        if (ns <= 1) return 0;
        const int last = ql * p.group - (nrb - 1) * kRows;
        return (nrb - 1) * kMergePerBlock + (last + kMergeRows - 1) / kMergeRows;
    };
    // group ids and merge offsets: exclusive scans over requests (contiguous ranges per thread)
    const int per = (a.R + kPlanThreads - 1) / kPlanThreads;
    const int r0 = min(a.R, tid * per), r1 = min(a.R, r0 + per);
    int mg = 0, mm = 0;
    for (int r = r0; r < r1; ++r) {
        int q0, ql, kv, ns, nrb;
        if (shape(r, q0, ql, kv, ns, nrb)) {
            mg += a.Hkv * ns;
            mm += a.Hkv * merges_of(ql, ns, nrb);
        }
    }
    int ig = mg, im = mm;
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const int tg = __shfl_up(ig, o, DSPARK_WAVE), tm = __shfl_up(im, o, DSPARK_WAVE);
        if (lane >= o) ig += tg, im += tm;
    }
    if (lane == DSPARK_WAVE - 1) s_wave[0][wave] = ig, s_wave[1][wave] = im;
    __syncthreads();
    int g0 = ig - mg, m0 = im - mm, mtot = 0;
    for (int w = 0; w < kPlanThreads / DSPARK_WAVE; ++w) {
        if (w < wave) g0 += s_wave[0][w], m0 += s_wave[1][w];
        mtot += s_wave[1][w];
    }
    for (int r = r0; r < r1; ++r) {
        int q0, ql, kv, ns, nrb;
        s_gid0[r] = g0;
        s_mb0[r] = m0;
        if (shape(r, q0, ql, kv, ns, nrb)) {
            g0 += a.Hkv * ns;
            m0 += a.Hkv * merges_of(ql, ns, nrb);
        }
    }
    __syncthreads();
    // histogram per queue and length: one thread per (request, split)
    const int S = p.max_splits;
    for (int u = tid; u < a.R * S; u += kPlanThreads) {
        const int r = u / S, sp = u - r * S;
        int q0, ql, kv, ns, nrb;
        if (!shape(r, q0, ql, kv, ns, nrb) || sp >= ns) continue;
        for (int g = 0; g < a.Hkv; ++g)
            atomicAdd(&s_bin[(s_gid0[r] + g * ns + sp) % kQueues][steps_of(kv, sp)], nrb);
    }
    __syncthreads();
    if (wave < kQueues) {
        // bin offsets of queue `wave`, longest first: lane l owns the bins at
        // descending positions kBinsPerLane * l .. kBinsPerLane * (l + 1) - 1
        int cnt[kBinsPerLane], mine = 0;
#pragma unroll
        for (int k = 0; k < kBinsPerLane; ++k) {
            const int bb = kBins - 1 - (kBinsPerLane * lane + k);
            cnt[k] = bb >= 0 ? s_bin[wave][bb] : 0;
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
            const int bb = kBins - 1 - (kBinsPerLane * lane + k);
            if (bb >= 0) s_bin[wave][bb] = run;
            run += cnt[k];
        }
        if (lane == DSPARK_WAVE - 1) s_qstart[wave] = incl;  // the queue's length, for now
    }
    __syncthreads();
    if (tid == 0) {
        int base = 0;
        for (int q = 0; q < kQueues; ++q) {
            const int len = s_qstart[q];
            p.head[q] = 0;
            p.head[kQueues + q] = base;
            p.head[2 * kQueues + q] = base + len;
            s_qstart[q] = base;
            base += len;
        }
        p.head[3 * kQueues] = mtot;
    }
    __syncthreads();
    // items: one thread per (request, split), the row blocks of a group together
    for (int u = tid; u < a.R * S; u += kPlanThreads) {
        const int r = u / S, sp = u - r * S;
        int q0, ql, kv, ns, nrb;
        if (!shape(r, q0, ql, kv, ns, nrb) || sp >= ns) continue;
        const int4 meta = int4{q0, ql, kv, ns};
        for (int g = 0; g < a.Hkv; ++g) {
            const int q = (s_gid0[r] + g * ns + sp) % kQueues;
            const int off = s_qstart[q] + atomicAdd(&s_bin[q][steps_of(kv, sp)], nrb);
            for (int b = 0; b < nrb; ++b) {
                p.list[2 * (off + b)] = int4{r, g, b, sp};
                p.list[2 * (off + b) + 1] = meta;
            }
        }
    }
    // merge items: one thread per (request, item); KV head, then row block, then rows
    const int M = a.Hkv * (p.rb_max * kMergePerBlock);  // items of a request, at most
    for (int u = tid; u < a.R * M; u += kPlanThreads) {
        const int r = u / M, j = u - r * M;
        int q0, ql, kv, ns, nrb;
        if (!shape(r, q0, ql, kv, ns, nrb)) continue;
        const int cnt = merges_of(ql, ns, nrb);
        if (j >= a.Hkv * cnt) continue;
        const int g = j / cnt, jj = j - g * cnt;
        const int off = s_mb0[r] + j;
        p.mlist[2 * off] = int4{r, g, jj / kMergePerBlock, kMergeRows * (jj % kMergePerBlock)};
        p.mlist[2 * off + 1] = int4{q0, ql, kv, ns};
    }
}

// ------------------------------------------------------------------ item

// LDS beside the copy ring: the probability exchange (double-buffered by step
// parity) and the per-row statistics.
struct Shared {
    uint2 p[2][kTilesPV][2][DSPARK_WAVE];  // [step parity][row tile][key block][lane]: 4 bf16
    float mx[kSW][kSTiles][16];            // row maxima per score wave
    float ls[kSW][kSTiles][16];            // row sums per score wave
    int lim[kSW];                          // per-wave minimum causal limit
    int item;                              // next work item (queue << 24 | index)
    int flag;                              // some row outgrew its reference
};

// Score role of one item (waves 0..3; sw = wave).  Barrier sequence per
// attempt: B0, [X in stage 0 of the first attempt], one per stage for stages
// 0 .. nsteps, then the two of the rerun check; the value role matches it.
__device__ __forceinline__ void score_item(const Params& p, const int r, const int g, const int rb,
                                           const int s, const int q0, const int ql, const int kv,
                                           const int nsplit, const uint32_t lds0, const int home,
                                           const int sw, int& nxt, Shared& sh) {
    const AttnArgs& a = p.a;
    constexpr int kSlotFloats = kRows * (kDv + 2);
    const int rows = ql * p.group;
    const int row0 = rb * kRows;
    int start, end;
    split_range(kv, s, start, end);
    const int nsteps = (end - start + kStep - 1) / kStep;  // >= 1
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const int hs = sw >> 1;  // row tiles 2 hs, 2 hs + 1
    const int kb = sw & 1;   // key block of every step
    const int partner = sw ^ 1;
    const uint16_t* __restrict__ qg = (const uint16_t*)a.q;

    // query fragments (B operand of S^T = K Q^T) and causal limits; rows past
    // the block's end get zero queries (finite scores, outputs never stored)
    bf16x8 qf[kSTiles][kKs];
    int lim[kSTiles];
    int lim_min = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < kSTiles; ++j) {
        const int row = row0 + 16 * (kSTiles * hs + j) + lr;
        if (row < rows) {
            const int t = row / p.group;
            const int h = g * p.group + (row - t * p.group);
            const uint16_t* qp = qg + ((int64_t)(q0 + t) * a.Hq + h) * kDk + 8 * lq;
#pragma unroll
            for (int ks = 0; ks < kKs; ++ks) qf[j][ks] = *(const bf16x8*)(qp + 32 * ks);
            lim[j] = kv - ql + t;
            lim_min = min(lim_min, lim[j]);
        } else {
#pragma unroll
            for (int ks = 0; ks < kKs; ++ks) qf[j][ks] = bf16x8{};
            lim[j] = -1;
        }
    }
    // the second tile's fragments live in the accumulation registers (free in
    // this role; the products read their B operand from there directly)
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks) asm volatile("" : "+a"(qf[1][ks]));
    lim_min = __reduce_min_sync(~0ull, lim_min);  // whole wave: a collective
    if (lane == 0) sh.lim[sw] = lim_min;          // read after the attempt's first barrier

    // mref: the row's fixed reference; mu: the same with -inf read as 0 (a row
    // that sees no key of the split); mobs: this lane's running maximum
    float mref[kSTiles], mu[kSTiles], mobs[kSTiles], lsum[kSTiles];
#pragma unroll
    for (int j = 0; j < kSTiles; ++j) mref[j] = mobs[j] = -__builtin_huge_valf();
    bool over = false;

    // K fragment offsets: rows 8 (lr / 4) + 4 kb + lr % 4, chunk 4 ks + lq
    uint32_t koff[2];
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
        const int t = 8 * (lr >> 2) + 4 * kb + (lr & 3);
        koff[kp] = lds0 + t * kRowB + pchunk(t, 4 * kp + lq) * 16;
    }

    auto compute = [&](int n, bool first_step, auto bufc) {
        constexpr unsigned buf = decltype(bufc)::value;
        constexpr uint32_t boff = buf * kTileB;
        const int tok0 = start + n * kStep;
        f32x4 sc[kSTiles][2];
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) sc[j][0] = sc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < kKs; ++ks) {
            const bf16x8 kf = *lds_ptr<const lds_bf16x8>(koff[ks & 1] + boff + 128 * (ks >> 1));
#pragma unroll
            for (int j = 0; j < kSTiles; ++j)
                sc[j][ks & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[j][ks], sc[j][ks & 1], 0, 0, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, kAheadK, 0);
#pragma unroll
        for (int i = 0; i < kKs - kAheadK; ++i) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, kSTiles, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, kSTiles * kAheadK, 0);
        __builtin_amdgcn_sched_barrier(0);

        // softmax over this wave's keys tok0 + 8 lq + 4 kb + e
        const bool full = tok0 + kStep <= end && tok0 + kStep - 1 <= lim_min;
        float sv[kSTiles][4], bm[kSTiles];
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) {
#pragma unroll
            for (int e = 0; e < 4; ++e) sv[j][e] = sc[j][0][e] + sc[j][1][e];
            if (!full) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int key = tok0 + 8 * lq + 4 * kb + e;
                    if (!(key < end && key <= lim[j])) sv[j][e] = -__builtin_huge_valf();
                }
            }
            // lane-local maximum: the reference is fixed, so a step needs the
            // row maximum across lanes only in the first step (and the
            // observed maximum once per item, reduced at the rerun check)
            bm[j] = vmax(vmax(sv[j][0], sv[j][1]), vmax(sv[j][2], sv[j][3])) * p.scale2;
            mobs[j] = vmax(mobs[j], bm[j]);
        }
        if (first_step) {
            // a row that sees no key of the first step sees none of the split
            // (its visible keys only grow), so its reference stays -inf
#pragma unroll
            for (int j = 0; j < kSTiles; ++j) bm[j] = row_max4(bm[j]);
            // the reference: the first step's maximum over both key blocks
            if (lq == 0) {
#pragma unroll
                for (int j = 0; j < kSTiles; ++j) sh.mx[sw][j][lr] = bm[j];
            }
            lds_barrier();  // X
#pragma unroll
            for (int j = 0; j < kSTiles; ++j) {
                mref[j] = vmax(bm[j], sh.mx[partner][j][lr]);
                mu[j] = mref[j] == -__builtin_huge_valf() ? 0.0f : mref[j];
            }
        }
        uint2* const pw = &sh.p[buf & 1][kSTiles * hs][kb][lane];
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) {
            over |= bm[j] > mref[j] + kRange;
            float pr[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) pr[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[j][e], p.scale2, -mu[j]));
            lsum[j] += (pr[0] + pr[1]) + (pr[2] + pr[3]);
            pw[j * 2 * DSPARK_WAVE] = uint2{cvt_pk_bf16(pr[0], pr[1]), cvt_pk_bf16(pr[2], pr[3])};
        }
    };

    const int claim = max(nsteps - 3, 0);
    for (int attempt = 0;; ++attempt) {
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) lsum[j] = 0.0f;
        lds_barrier();  // B0: step 0 in LDS; sh.lim written
        if (attempt == 0) lim_min = min(min(sh.lim[0], sh.lim[1]), min(sh.lim[2], sh.lim[3]));
        auto one = [&](int n, auto bufc) {
            if (n == claim && tid == 0 && attempt == 0) nxt = atomicAdd(p.head + home, 1);
            compute(n, n == 0 && attempt == 0, bufc);
            lds_barrier();  // end of stage n
        };
        for (int n = 0; n < nsteps; n += kRing) {
            one(n, std::integral_constant<unsigned, 0>{});
            if (n + 1 < nsteps) one(n + 1, std::integral_constant<unsigned, 1>{});
            if (n + 2 < nsteps) one(n + 2, std::integral_constant<unsigned, 2>{});
            if (n + 3 < nsteps) one(n + 3, std::integral_constant<unsigned, 3>{});
        }
        lds_barrier();  // end of stage nsteps (the value waves' last product)
        // rerun check: did any row outgrow its reference?  (ballot on the whole wave)
        const bool any_over = __builtin_amdgcn_ballot_w64(over) != 0;
        if (lane == 0 && any_over) atomicOr(&sh.flag, 1);
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) mobs[j] = row_max4(mobs[j]);
        if (lq == 0) {
#pragma unroll
            for (int j = 0; j < kSTiles; ++j) sh.mx[sw][j][lr] = mobs[j];
        }
        __syncthreads();
        const int again = sh.flag;
        float mnext[kSTiles];
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) mnext[j] = vmax(mobs[j], sh.mx[partner][j][lr]);
        __syncthreads();
        if (!again) break;
        if (tid == 0) sh.flag = 0;
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) {
            mref[j] = mnext[j];
            mu[j] = mref[j] == -__builtin_huge_valf() ? 0.0f : mref[j];
        }
        over = false;
    }

    // row sums over the four lanes of a row; the pair's halves are added by the readers
#pragma unroll
    for (int j = 0; j < kSTiles; ++j) {
        lsum[j] += __shfl_xor(lsum[j], 16, 64);
        lsum[j] += __shfl_xor(lsum[j], 32, 64);
    }
    if (lq == 0) {
#pragma unroll
        for (int j = 0; j < kSTiles; ++j) sh.ls[sw][j][lr] = lsum[j];
    }
    __syncthreads();  // F: the value waves read the sums next
    if (kb != 0 || lq != 0) return;
    // waves 0 and 2 write the statistics of their two row tiles
#pragma unroll
    for (int j = 0; j < kSTiles; ++j) {
        const int rr = 16 * (kSTiles * hs + j) + lr;
        if (row0 + rr >= rows) continue;
        const float L = sh.ls[sw][j][lr] + sh.ls[partner][j][lr];
        if (nsplit == 1) {
            if (a.lse) {
                const int row = row0 + rr;
                const int t = row / p.group;
                const int h = g * p.group + (row - t * p.group);
                a.lse[(int64_t)(q0 + t) * a.Hq + h] = (mref[j] + log2f(L)) * kLn2;
            }
        } else {
            float* part = p.part + (((int64_t)(r * a.Hkv + g) * p.rb_max + rb) * p.max_splits + s) * kSlotFloats;
            part[rr] = mref[j];
            part[kRows + rr] = L;
        }
    }
}

// Value role of one item (waves 4..7; vw = wave - 4): the copies and the
// value product, on the score role's barrier sequence.
__device__ __forceinline__ void value_item(const Params& p, const int r, const int g, const int rb,
                                           const int s, const int q0, const int ql, const int kv,
                                           const int nsplit, const uint32_t lds0, const int vw,
                                           Shared& sh) {
    const AttnArgs& a = p.a;
    constexpr int kSlotFloats = kRows * (kDv + 2);
    const int rows = ql * p.group;
    const int row0 = rb * kRows;
    int start, end;
    split_range(kv, s, start, end);
    const int nsteps = (end - start + kStep - 1) / kStep;  // >= 1
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const uint16_t* __restrict__ kc = (const uint16_t*)a.k;

    // page ids of the split, kPageRegs per lane
    const int pg0 = start >> p.page_shift;
    const int npg = ((end - 1) >> p.page_shift) - pg0 + 1;
    int my_page[kPageRegs];
#pragma unroll
    for (int k = 0; k < kPageRegs; ++k) {
        const int i = k * DSPARK_WAVE + lane;
        my_page[k] = i < npg ? a.block_table[(int64_t)r * a.max_pages + pg0 + i] : 0;
    }

    // V^T fragment offsets (transposing reads): rows 8 lq + 4 h + lr / 4, chunk
    // 2 db + (lr % 4) / 2, half lr % 2, for this wave's blocks db = 8 vw + d
    uint32_t voff[4][2];
#pragma unroll
    for (int dq = 0; dq < 4; ++dq)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int t = 8 * lq + 4 * h + (lr >> 2);
            const int c = 2 * dq + ((lr & 3) >> 1);
            voff[dq][h] = lds0 + t * kRowB + pchunk(t, c) * 16 + (lr & 1) * 8 + 256 * vw;
        }

    // copy geometry: this wave's copy instructions cover tile chunks
    // (first + i) * 64 + lane, row / 72, physical chunk % 72
    const int first = kCopies * vw;
    auto cp_at = [&](int i, int ln, int& t, int& c) {
        const int pp_ = (first + i) * 64 + ln;
        t = pp_ / kRowChunks;
        c = pchunk(t, pp_ - t * kRowChunks);
    };
    const uint64_t kc_head = (uint64_t)(uintptr_t)kc + (uint64_t)((uint32_t)g * p.s1b);
    const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds0 + first * 1024);
    auto page_of = [&](int idx) {
        int pg = 0;
#pragma unroll
        for (int k = 0; k < kPageRegs; ++k)
            if ((idx >> 6) == k) pg = __builtin_amdgcn_readlane(my_page[k], idx & 63);
        return pg;
    };
    uint32_t cpo[kCopies];
#pragma unroll
    for (int i = 0; i < kCopies; ++i) {
        int t, c;
        cp_at(i, lane, t, c);
        cpo[i] = t * p.s2b + 16 * c;
    }
    auto issue = [&](int n) {
        const int tok0 = start + n * kStep;
        const int pidx = min(max((tok0 >> p.page_shift) - pg0, 0), kPageRegs * DSPARK_WAVE - 1);
        const int page = page_of(pidx);
        const int slot0 = tok0 & ((1 << p.page_shift) - 1);
        const uint32_t dst = lds_wave + ((unsigned)n % kRing) * kTileB;
        if (tok0 + kStep <= end) {
            const uint64_t kbase = kc_head + (uint64_t)(uint32_t)page * p.s0b + (uint32_t)slot0 * p.s2b;
#pragma unroll
            for (int i = 0; i < kCopies; ++i) lds_copy16_s(kbase, cpo[i], dst + i * 1024);
        } else {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            // last, partial step or past the end: keys at or past the end read the zero row
            const uint16_t* kbase = kc + (int64_t)page * a.ks[0] + (int64_t)g * a.ks[1];
#pragma unroll
            for (int i = 0; i < kCopies; ++i) {
                int t, c;
                cp_at(i, ln, t, c);
                const bool in = tok0 + t < end;
                const uint16_t* src = in ? kbase + (int64_t)(slot0 + t) * a.ks[2] + 8 * c : g_zero_row + 8 * c;
                lds_copy16(src, dst + i * 1024);
            }
        }
    };

    f32x4 acc[kTilesPV][kDbW];
    auto product = [&](auto bufc) {
        constexpr unsigned buf = decltype(bufc)::value;
        constexpr uint32_t boff = buf * kTileB;
        __builtin_amdgcn_sched_barrier(0);
        const uint2* const pr0 = &sh.p[buf & 1][0][0][lane];
        bf16x8 pf[kTilesPV];
#pragma unroll
        for (int ti = 0; ti < kTilesPV; ++ti) {
            const uint2 lo = pr0[ti * 2 * DSPARK_WAVE];
            const uint2 hi = pr0[ti * 2 * DSPARK_WAVE + DSPARK_WAVE];
            pf[ti] = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
        }
#pragma unroll
        for (int d = 0; d < kDbW; ++d) {
            const uint32_t vo = boff + 128 * (d >> 2);
            const s16x4 h0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(lds_ptr<lds_s16x4>(voff[d & 3][0] + vo));
            const s16x4 h1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(lds_ptr<lds_s16x4>(voff[d & 3][1] + vo));
            const bf16x8 vf = __builtin_bit_cast(
                bf16x8, (short __attribute__((ext_vector_type(8)))){h0[0], h0[1], h0[2], h0[3],
                                                                     h1[0], h1[1], h1[2], h1[3]});
#pragma unroll
            for (int ti = 0; ti < kTilesPV; ++ti)
                acc[ti][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[ti], acc[ti][d], 0, 0, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * kTilesPV + kAheadV, 0);
#pragma unroll
        for (int i = 0; i < kDbW - kAheadV / 2; ++i) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, kTilesPV, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, kTilesPV * kAheadV / 2, 0);
        __builtin_amdgcn_sched_barrier(0);
    };

    for (int attempt = 0;; ++attempt) {
        // the accumulators live in the accumulation registers (the score role
        // keeps its second query tile there; this role's vector registers hold
        // the operand pipeline)
#pragma unroll
        for (int ti = 0; ti < kTilesPV; ++ti)
#pragma unroll
            for (int d = 0; d < kDbW; ++d) {
                acc[ti][d] = f32x4{0.f, 0.f, 0.f, 0.f};
                asm volatile("" : "+a"(acc[ti][d]));
            }
        // every thread issues kCopies copies per step, in order, also past the
        // last step (zero-row copies into buffers not read again), so "step n
        // has landed" is vmcnt <= kCopies once step n + 1 is issued
        wait_vmcnt<0>();
        issue(0);
        issue(1);
        wait_vmcnt<kCopies>();
        lds_barrier();  // B0
        // stage t: copies of step t + 2, then the product of step t - 1
        auto one = [&](int t, auto bufc) {
            issue(t + 2);
            if (t == 0 && attempt == 0) lds_barrier();  // X (the score waves' reference exchange)
            if (t >= 1) product(bufc);
            wait_vmcnt<kCopies>();  // step t + 1 has landed
            lds_barrier();          // end of stage t
        };
        for (int t = 0; t <= nsteps; t += kRing) {
            // stage t reads step t - 1, in buffer (t - 1) % 4
            one(t, std::integral_constant<unsigned, 3>{});
            if (t + 1 <= nsteps) one(t + 1, std::integral_constant<unsigned, 0>{});
            if (t + 2 <= nsteps) one(t + 2, std::integral_constant<unsigned, 1>{});
            if (t + 3 <= nsteps) one(t + 3, std::integral_constant<unsigned, 2>{});
        }
        wait_vmcnt<0>();
        __syncthreads();
        const int again = sh.flag;
        __syncthreads();
        if (!again) break;
    }

    __syncthreads();  // F: the score waves' row sums are in LDS
    float L[kTilesPV];
#pragma unroll
    for (int ti = 0; ti < kTilesPV; ++ti) {
        const int w0 = 2 * (ti / kSTiles);
        L[ti] = sh.ls[w0][ti % kSTiles][lr] + sh.ls[w0 + 1][ti % kSTiles][lr];
    }
    if (nsplit == 1) {
        uint16_t* outp = (uint16_t*)a.out;
#pragma unroll
        for (int ti = 0; ti < kTilesPV; ++ti) {
            const int row = row0 + 16 * ti + lr;
            if (row < rows) {
                const int t = row / p.group;
                const int h = g * p.group + (row - t * p.group);
                const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
                const float inv = 1.0f / L[ti];
#pragma unroll
                for (int d = 0; d < kDbW; ++d) {
                    uint2 pk;
                    pk.x = pack2_bf16(acc[ti][d][0] * inv, acc[ti][d][1] * inv);
                    pk.y = pack2_bf16(acc[ti][d][2] * inv, acc[ti][d][3] * inv);
                    *(uint2*)(outp + orow * kDv + 16 * (kDbW * vw + d) + 4 * lq) = pk;
                }
            }
        }
        return;
    }
    float* part = p.part + (((int64_t)(r * a.Hkv + g) * p.rb_max + rb) * p.max_splits + s) * kSlotFloats;
#pragma unroll
    for (int ti = 0; ti < kTilesPV; ++ti) {
        const int rr = 16 * ti + lr;
        if (row0 + rr < rows) {
#pragma unroll
            for (int d = 0; d < kDbW; ++d)
                *(f32x4*)(part + 2 * kRows + rr * kDv + 16 * (kDbW * vw + d) + 4 * lq) = acc[ti][d];
        }
    }
}

// Persistent workgroups of eight waves: workgroup b serves queue b % 8 (its
// XCD), then the others.  Each role runs its own item loop; the loops meet at
// the same barriers.
__global__ __launch_bounds__(kThreads) void mla_kernel(Params p) {
    __shared__ __align__(16) unsigned char lds[kRing * kTileB];
    __shared__ Shared sh;
    uint32_t lds0 = (uint32_t)(uintptr_t)&lds[0];
    asm volatile("" : "+s"(lds0));
    const int home0 = blockIdx.x % kQueues;
    auto claim_any = [&](int q_first) {
        for (int k = 0; k < kQueues; ++k) {
            const int q = (q_first + k) % kQueues;
            const int c = atomicAdd(p.head + q, 1);
            if (p.head[kQueues + q] + c < p.head[2 * kQueues + q]) return (q << 24) | c;
        }
        return -1;
    };
    if (threadIdx.x == 0) {
        sh.flag = 0;
        sh.item = claim_any(home0);
    }
    __syncthreads();
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    int cur = __builtin_amdgcn_readfirstlane(sh.item);
    if (wave < kSW) {
        while (cur >= 0) {
            const int q = cur >> 24;
            const int it = p.head[kQueues + q] + (cur & 0xffffff);
            const int4 e0 = p.list[2 * it];
            const int4 e1 = p.list[2 * it + 1];
            int nxt = 0;  // index claimed from queue q near the end of the item (thread 0)
            score_item(p, e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w, lds0, q, wave, nxt, sh);
            __syncthreads();
            if (threadIdx.x == 0) {
                sh.item = p.head[kQueues + q] + nxt < p.head[2 * kQueues + q] ? (q << 24) | nxt
                                                                               : claim_any(q + 1);
            }
            __syncthreads();
            cur = __builtin_amdgcn_readfirstlane(sh.item);
        }
    } else {
        while (cur >= 0) {
            const int q = cur >> 24;
            const int it = p.head[kQueues + q] + (cur & 0xffffff);
            const int4 e0 = p.list[2 * it];
            const int4 e1 = p.list[2 * it + 1];
            value_item(p, e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w, lds0, wave - kSW, sh);
            __syncthreads();
            __syncthreads();
            cur = __builtin_amdgcn_readfirstlane(sh.item);
        }
    }
}

// Combines the split partials of kMergeRows rows: 64 threads per row, eight
// output dims each, splits in index order.
constexpr int kMergeBatch = 8;
__global__ __launch_bounds__(256) void mla_merge(Params p) {
    constexpr int kSlotFloats = kRows * (kDv + 2);
    const AttnArgs& a = p.a;
    const int count = p.head[3 * kQueues];
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
        const int r = e0.x, g = e0.y, rb = e0.z;
        const int q0 = e1.x, ql = e1.y, ns = e1.w;
        const int rows = ql * p.group;
        const int nrows = min(kRows, rows - rb * kRows);
        const int mr = e0.w + (tid >> 6);
        if (mr >= nrows) continue;
        const int c8 = (tid & 63) * 8;
        const float* base = p.part + ((int64_t)(r * a.Hkv + g) * p.rb_max + rb) * p.max_splits * kSlotFloats;
        float M = -__builtin_huge_valf(), L = 0.0f;
        f32x4 o0 = f32x4{0.f, 0.f, 0.f, 0.f}, o1 = o0;
        for (int s0 = 0; s0 < ns; s0 += kMergeBatch) {
            float ms[kMergeBatch], ls[kMergeBatch];
            f32x4 a0[kMergeBatch], a1[kMergeBatch];
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const float* sl = base + (int64_t)min(s0 + k, ns - 1) * kSlotFloats;
                ms[k] = sl[mr];
                ls[k] = sl[kRows + mr];
                a0[k] = *(const f32x4*)(sl + 2 * kRows + mr * kDv + c8);
                a1[k] = *(const f32x4*)(sl + 2 * kRows + mr * kDv + c8 + 4);
            }
            float Mb = M;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k)
                if (s0 + k < ns) Mb = fmaxf(Mb, ms[k]);
            if (M > -__builtin_huge_valf() && Mb != M) {
                const float f = exp2f(M - Mb);
                L *= f;
                o0 *= f;
                o1 *= f;
            }
            M = Mb;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                if (s0 + k >= ns) break;
                const float f = ms[k] > -__builtin_huge_valf() ? exp2f(ms[k] - M) : 0.0f;
                L += ls[k] * f;
                o0 += f * a0[k];
                o1 += f * a1[k];
            }
        }
        const int row = rb * kRows + mr;
        const int t = row / p.group;
        const int h = g * p.group + (row - t * p.group);
        const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
        const float inv = 1.0f / L;
        uint4 pk;
        pk.x = pack2_bf16(o0[0] * inv, o0[1] * inv);
        pk.y = pack2_bf16(o0[2] * inv, o0[3] * inv);
        pk.z = pack2_bf16(o1[0] * inv, o1[1] * inv);
        pk.w = pack2_bf16(o1[2] * inv, o1[3] * inv);
        *(uint4*)((uint16_t*)a.out + orow * kDv + c8) = pk;
        if (a.lse && c8 == 0) a.lse[orow] = (M + log2f(L)) * kLn2;
    }
}

}  // namespace mla

bool attn_mla_shape_ok(const AttnArgs& a) {
    return a.bf16 && a.Dqk == mla::kDk && a.Dv == mla::kDv && a.Hq % a.Hkv == 0 &&
           a.page >= 64 && (a.page & (a.page - 1)) == 0;
}

bool attn_mla_supported(const AttnArgs& a) {
    const int64_t lim = (int64_t)1 << 30;
    // values must be the first Dv dims of the key rows
    return attn_mla_shape_ok(a) && a.v == a.k && a.vs[0] == a.ks[0] && a.vs[1] == a.ks[1] &&
           a.vs[2] == a.ks[2] && a.ks[0] < lim && a.ks[1] < lim && a.ks[2] < lim &&
           a.ks[0] % 8 == 0 && a.ks[1] % 8 == 0 && a.ks[2] % 8 == 0 &&
           ((uintptr_t)a.q % 16) == 0 && ((uintptr_t)a.k % 16) == 0 && ((uintptr_t)a.out % 16) == 0;
}

size_t attn_mla_workspace(const AttnArgs& a) {
    const mla::Geom g = mla::geom(a);
    return g.head_bytes + g.list_bytes + g.mlist_bytes + g.part_bytes;
}

hipError_t launch_attn_mla(const AttnArgs& a, void* ws, hipStream_t s) {
    const mla::Geom g = mla::geom(a);
    mla::Params p;
    p.a = a;
    p.group = g.group;
    p.rb_max = g.rb_max;
    p.max_splits = g.max_splits;
    p.page_shift = __builtin_ctz((unsigned)a.page);
    p.s0b = (uint32_t)(a.ks[0] * 2);
    p.s1b = (uint32_t)(a.ks[1] * 2);
    p.s2b = (uint32_t)(a.ks[2] * 2);
    p.scale2 = a.scale * mla::kLog2e;
    p.head = (int*)ws;
    p.list = (int4*)((char*)ws + g.head_bytes);
    p.mlist = (int4*)((char*)ws + g.head_bytes + g.list_bytes);
    p.part = (float*)((char*)ws + g.head_bytes + g.list_bytes + g.mlist_bytes);
    hipLaunchKernelGGL(mla::mla_plan, dim3(1), dim3(mla::kPlanThreads), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // one workgroup per CU (157 KB of LDS, eight waves: two per SIMD)
    const int64_t grid = std::min<int64_t>(cus, std::max<int64_t>(g.n_items, 1));
    hipLaunchKernelGGL(mla::mla_kernel, dim3((unsigned)grid), dim3(mla::kThreads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess || g.n_merge == 0) return e;
    const int64_t mgrid = std::min<int64_t>((int64_t)cus * 16, g.n_merge);
    hipLaunchKernelGGL(mla::mla_merge, dim3((unsigned)mgrid), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace dspark

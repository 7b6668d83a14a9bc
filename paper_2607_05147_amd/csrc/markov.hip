// Markov-head draft block on gfx950: the drafter's sequential stage.
//
// For every request r, with x_0 = anchor[r] and k = 1 .. K (the left-to-right
// factorisation of the semi-autoregressive stage, eq. sequential-factorization,
// with the Markov head's low-rank transition bias of eq. markov, and the
// confidence head of eq. confidence with the per-position temperatures of its
// post-hoc calibration):
//   e_k = W1[x_{k-1}];   z_k = inv_temp * (U_k + W2^T e_k);   p_k = softmax(z_k);
//   x_k = inverse CDF of p_k at u[r, k-1];   c_k = sigmoid(w . [h_k; e_k] / T_k).
// Launches, all on one stream: md_hidden (the backbone part w_h . h_k of every
// confidence logit, once) and md_first (e_1 and c_1), then per position k
// either one md_coop launch per group of up to 128 requests (bf16 base
// logits, V % 4 == 0, a grid the device holds at once; md_check after the
// block), which keeps z in registers across two grid-wide
// exchanges so that the projection and the base logits are read once and p
// is written once, or the three launches:
//   md_tile   one workgroup per 128 vocabulary entries: W2^T e for every
//             request on v_mfma_f32_16x16x32_bf16 (the tile's W2t rows stay in
//             registers as A operands, the embeddings stream through LDS in
//             chunks of 32 requests as B operands), plus the base logits; z is
//             written to draft_p in fp32, with the tile's softmax statistics
//             (max, sum of exp) per request;
//   md_stats  one wave per request: the row's max and total and the tile in
//             which the running mass passes u * total (fp64 prefix over the
//             tiles in vocabulary order);
//   md_norm   a streaming pass over draft_p that turns z into
//             p_k = exp(z - max) / total in place; the workgroup whose segment
//             holds a request's draw makes it (fp64 prefix of that tile's
//             masses), writes x_k, gathers e_{k+1} into the other embedding
//             buffer and writes c_{k+1}.
// The positions of a block are sequential by definition (x_k feeds position
// k + 1).
#include <algorithm>
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace dspark {
namespace mkd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / DSPARK_WAVE;
constexpr int kTileV = 128;              // vocabulary entries per workgroup tile
constexpr int kWaveV = kTileV / kWaves;  // 32 per wave
constexpr int kVT = kWaveV / 16;         // 16-entry blocks per wave
constexpr int kChunkR = 32;              // requests per LDS chunk
constexpr int kRT = kChunkR / 16;        // 16-request blocks per chunk

__host__ __device__ constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// md_coop's grid barrier: arrival groups of workgroups (blockIdx % 8) and its
// words in the workspace, 128 bytes apart: [0] arrivals of the groups' last
// workgroups, [1] timeout, [stride * (1 + x)] arrivals of group x,
// [stride * (1 + groups + x)] flag of group x
constexpr int kCoGroups = 8;
constexpr int kSyncStride = 32;
constexpr int kSyncWords = kSyncStride * (1 + 2 * kCoGroups);

// Slot of 16-byte chunk c in row t of the embedding chunk (nch chunks per row,
// a power of two).  The XOR (bits of t in the order 0, 2, 1, 3) puts the 16
// lanes of every phase of the B-operand reads on distinct banks for every
// supported rank (gfx950 serves a 16-byte LDS read in four 16-lane phases split
// by lane bit 5 and the parity of lane bits 2 ^ 3 ^ 4).
__device__ __forceinline__ int eslot(int t, int c, int nch) {
    const int f = (t & 1) | (((t >> 2) & 1) << 1) | (((t >> 1) & 1) << 2) | (((t >> 3) & 1) << 3);
    return c ^ (f & (nch - 1));
}

// token of position k - 1 (the anchor for k = 1); -1 when it is not a valid token
__device__ __forceinline__ int prev_token(const MarkovArgs& a, int r, int k) {
    const int x = k == 1 ? a.anchor[r] : a.draft_tok[(int64_t)r * a.K + (k - 2)];
    return x >= 0 && x < a.V ? x : -1;
}

// Maximum / sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the lanes that
// hold one request's entries of a block), with lane swaps instead of LDS.
__device__ __forceinline__ float quad_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Per-request state of a position, from the tile statistics to the normalisation.
struct RowInfo {
    float M;     // row maximum of z (base-2 units: z * log2 e)
    float S;     // sum over the row of exp(z - M)
    int tile;    // tile in which the running mass passes u * S
    int pad;
    double thr;  // u * S minus the mass of the tiles before `tile` (+inf: the tile's last entry with mass)
};

// w_e . W1[x] over one wave (every lane gets the sum)
__device__ __forceinline__ float embed_dot(const MarkovArgs& a, const uint16_t* w1, int lane) {
    float s = 0.0f;
    for (int j = lane; j < a.rank; j += DSPARK_WAVE) s += a.w_conf[a.d + j] * bf16_to_f32(w1[j]);
    return wave_sum(s);
}

__device__ __forceinline__ float confidence(const MarkovArgs& a, float logit, int k) {
    const float T = a.sts_temp ? a.sts_temp[k - 1] : 1.0f;
    return 1.0f / (1.0f + expf(-logit / T));
}

// --------------------------------------------------------------- md_hidden

// The backbone part of every confidence logit, w_h . h_k, for all (r, k):
// one wave per row (independent of the drawn tokens, so done once up front).
__global__ __launch_bounds__(kThreads) void md_hidden(MarkovArgs a, float* sh) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * kWaves + wave;
    if (row >= (int64_t)a.R * a.K) return;  // whole wave
    const uint16_t* h = a.hidden + row * a.d;
    float s = 0.0f;
    if ((a.d & 7) == 0 && ((uintptr_t)a.hidden & 15) == 0) {
        for (int i = lane * 8; i < a.d; i += DSPARK_WAVE * 8) {
            const uint4 hv = *(const uint4*)(h + i);
            const uint32_t w4[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
            for (int q = 0; q < 4; ++q)
                s += a.w_conf[i + 2 * q] * __uint_as_float(w4[q] << 16) +
                     a.w_conf[i + 2 * q + 1] * __uint_as_float(w4[q] & 0xffff0000u);
        }
    } else {
        for (int i = lane; i < a.d; i += DSPARK_WAVE) s += a.w_conf[i] * bf16_to_f32(h[i]);
    }
    s = wave_sum(s);
    if (lane == 0) sh[row] = s;
}

// ---------------------------------------------------------------- md_first

// Position 1: e_1 = W1[x_0] into the first embedding buffer, and c_1.  One wave per request.
// Also zeroes md_coop's barrier words (when given).
__global__ __launch_bounds__(kThreads) void md_first(MarkovArgs a, const float* sh, uint16_t* E0, unsigned* sync) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (sync && blockIdx.x == 0)
        for (int i = threadIdx.x; i < kSyncWords; i += kThreads) sync[i] = 0u;
    const int r = blockIdx.x * kWaves + wave;
    if (r >= a.R) return;  // whole wave
    const int x0 = a.anchor[r];
    const bool ok = x0 >= 0 && x0 < a.V;
    const uint16_t* w1 = a.W1 + (int64_t)(ok ? x0 : 0) * a.rank;
    for (int j = lane * 8; j < a.rank; j += DSPARK_WAVE * 8)
        *(uint4*)(E0 + (int64_t)r * a.rank + j) = *(const uint4*)(w1 + j);
    const float s = embed_dot(a, w1, lane) + (sh ? sh[(int64_t)r * a.K] : 0.0f);
    if (lane == 0) a.conf[(int64_t)r * a.K] = ok ? confidence(a, s, 1) : __builtin_nanf("");
}

// ----------------------------------------------------------------- md_tile

// z for (request, vocabulary entry) pairs of one 128-entry tile:
// C[v, r] = sum_j W2t[v, j] E[r, j] on MFMA (A: the tile's W2t rows, kept in
// registers; B: the embeddings, 32 requests at a time through LDS), then
// z = inv_temp * (U + C), kept in base-2 units (z * log2 e, so that exp(z - m)
// is one v_exp_f32 of the difference).  z goes to the request's draft_p row
// (md_norm turns it into p in place), and the per-tile statistics to
// stats[r * ntiles + tile] = (max z, sum 2^(z - max)).
// VEC: 4 consecutive entries per lane are loaded / stored as one vector
// (V, ld multiples of 4, aligned rows).
// NT: bf16 terms of the B operand per request (1: the embedding itself; 2:
// the RNN head's fp32 output split as hi + mid, the second term the bf16
// rounding of what the first leaves, so the products see the fp32 vector to
// within 2^-16 of each entry); E row r holds the NT terms one after the other.
// BF16: the base logits' type.  Their loads are branch-free (clamped
// indices; entries past V are masked with the rest of the tile), so they issue
// back to back and stay in flight during the products.  Occupancy: three
// waves per SIMD for one term; two for more terms (more staged embedding
// loads), which leaves their loads room without spilling (measured faster
// with three terms).
template <int KS, int NT, bool VEC, bool BF16>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(NT == 1 ? 3 : 2, 4))) void md_tile(
    MarkovArgs a, const uint16_t* E, float2* stats, int ntiles, int k) {
    constexpr int kNch = 4 * KS;  // 16-byte chunks per embedding row
    constexpr int kRank = 32 * KS;
    __shared__ __align__(16) uint16_t se[NT * kChunkR * kRank];
    __shared__ float2 sst[kWaves][kChunkR];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const int tile = blockIdx.x;
    const int v0 = tile * kTileV + wave * kWaveV;
    constexpr float kLog2e = 1.4426950408889634f;
    const float scale2 = a.inv_temp * kLog2e;

    // A fragments: W2t rows v0 + 16 vt + lr (clamped into the vocabulary), dims 32 ks + 8 lq ..
    bf16x8 af[kVT][KS];
#pragma unroll
    for (int vt = 0; vt < kVT; ++vt) {
        const int v = min(v0 + 16 * vt + lr, a.V - 1);
        const uint16_t* src = a.W2t + (int64_t)v * kRank + 8 * lq;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) af[vt][ks] = *(const bf16x8*)(src + 32 * ks);
    }

    for (int c0 = 0; c0 < a.R; c0 += kChunkR) {
        const bool interior = (tile + 1) * kTileV <= a.V && c0 + kChunkR <= a.R;
        // the chunk's embeddings first, then its base logits: the LDS stores
        // below wait only for the embeddings (loads complete in order), and the
        // base logits stay in flight during the products
        // (measured: this guarded form schedules better than clamped, unguarded
        // loads, by 1.4x on a three-term product)
        constexpr int kCopy = ceil_div(NT * kChunkR * kNch, kThreads);
        uint4 ev[kCopy];
#pragma unroll
        for (int i = 0; i < kCopy; ++i) {
            const int idx = tid + i * kThreads;  // (request t, term, chunk)
            const int t = idx / (NT * kNch);
            ev[i] = idx < NT * kChunkR * kNch && c0 + t < a.R
                        ? *(const uint4*)(E + (int64_t)(c0 + t) * (NT * kRank) + 8 * (idx % (NT * kNch)))
                        : uint4{0u, 0u, 0u, 0u};
        }
        float ub[kRT][kVT][4];
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int r = min(c0 + 16 * rt + lr, a.R - 1);
            const int64_t row = (int64_t)r * a.K + (k - 1);
#pragma unroll
            for (int vt = 0; vt < kVT; ++vt) {
                const int vb = v0 + 16 * vt + 4 * lq;
                if (VEC) {
                    // V % 4 == 0: a group below V lies wholly inside the row
                    const int vc = min(vb, a.V - 4);
                    if (BF16) {
                        const uint2 w = *(const uint2*)((const uint16_t*)a.base + row * a.ld + vc);
                        ub[rt][vt][0] = __uint_as_float(w.x << 16);
                        ub[rt][vt][1] = __uint_as_float(w.x & 0xffff0000u);
                        ub[rt][vt][2] = __uint_as_float(w.y << 16);
                        ub[rt][vt][3] = __uint_as_float(w.y & 0xffff0000u);
                    } else {
                        const float4 w = *(const float4*)((const float*)a.base + row * a.ld + vc);
                        ub[rt][vt][0] = w.x, ub[rt][vt][1] = w.y, ub[rt][vt][2] = w.z, ub[rt][vt][3] = w.w;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int64_t i = row * a.ld + min(vb + e, a.V - 1);
                        ub[rt][vt][e] = BF16 ? bf16_to_f32(((const uint16_t*)a.base)[i]) : ((const float*)a.base)[i];
                    }
                }
            }
        }
        lds_barrier();  // the previous chunk's LDS reads are done (global loads stay in flight)
        // (no guard when the copy divides evenly: a branch here would make the
        // stores wait for the base logits as well)
        constexpr bool kExact = NT * kChunkR * kNch % kThreads == 0;
#pragma unroll
        for (int i = 0; i < kCopy; ++i) {
            const int idx = tid + i * kThreads;
            const int t = idx / (NT * kNch), nt = (idx / kNch) % NT, c = idx % kNch;
            if (kExact || idx < NT * kChunkR * kNch)
                *(uint4*)(se + ((nt * kChunkR + t) * kNch + eslot(t, c, kNch)) * 8) = ev[i];
        }
        lds_barrier();

        // lane holds C[v, r] for v = v0 + 16 vt + 4 lq + e, r = c0 + 16 rt + lr
        f32x4 acc[kVT][kRT];
#pragma unroll
        for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) acc[vt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int t = 16 * rt + lr;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 b =
                        *(const bf16x8*)(se + ((nt * kChunkR + t) * kNch + eslot(t, 4 * ks + lq, kNch)) * 8);
#pragma unroll
                    for (int vt = 0; vt < kVT; ++vt)
                        acc[vt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[vt][ks], b, acc[vt][rt], 0, 0, 0);
                }
        }

#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const int r = c0 + 16 * rt + lr;
            const bool rok = r < a.R;
            float z[kVT][4];
#pragma unroll
            for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                for (int e = 0; e < 4; ++e) z[vt][e] = scale2 * (ub[rt][vt][e] + acc[vt][rt][e]);
            if (!interior) {  // the vocabulary's last tile or the requests' last chunk
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (!(rok && v0 + 16 * vt + 4 * lq + e < a.V)) z[vt][e] = -__builtin_huge_valf();
            }
            if (rok) {  // z itself, normalised in place by md_norm
                float* out = a.draft_p + ((int64_t)r * a.K + (k - 1)) * a.V;
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt) {
                    const int vb = v0 + 16 * vt + 4 * lq;
                    if (VEC && vb + 3 < a.V) {
                        *(float4*)(out + vb) = float4{z[vt][0], z[vt][1], z[vt][2], z[vt][3]};
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (vb + e < a.V) out[vb + e] = z[vt][e];
                    }
                }
            }
            float m = -__builtin_huge_valf();
#pragma unroll
            for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                for (int e = 0; e < 4; ++e) m = fmaxf(m, z[vt][e]);
            m = quad_max(m);
            float s = 0.0f;
            if (m > -__builtin_huge_valf()) {
#pragma unroll
                for (int vt = 0; vt < kVT; ++vt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) s += __builtin_amdgcn_exp2f(z[vt][e] - m);
            }
            s = quad_sum(s);
            if (lq == 0) sst[wave][16 * rt + lr] = float2{m, s};
        }
        lds_barrier();
        if (tid < kChunkR && c0 + tid < a.R) {
            float M = -__builtin_huge_valf();
#pragma unroll
            for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sst[w][tid].x);
            float S = 0.0f;
            if (M > -__builtin_huge_valf()) {
#pragma unroll
                for (int w = 0; w < kWaves; ++w)
                    if (sst[w][tid].x > -__builtin_huge_valf()) S += sst[w][tid].y * exp2f(sst[w][tid].x - M);
            }
            stats[(int64_t)(c0 + tid) * ntiles + tile] = float2{M, S};
        }
    }
}

// ---------------------------------------------------------------- md_stats

// Per request (one wave): the row maximum and total from the tile statistics
// (tile masses in fp64), and the tile in which the running mass passes
// u * total, scanning the tiles in vocabulary order.  Lane l takes the
// contiguous run of tiles l * per .. l * per + per - 1, so the lane order is
// the vocabulary order; the reductions are lane shuffles, with no barrier.
constexpr int kStatsMaxPer = 32;  // tiles per lane (up to 2048 tiles: V <= 262144)
// Device-coherent 64-bit access (agent scope, relaxed): it bypasses the
// per-XCD L2, for data that the workgroups of one cooperative launch exchange
// across a grid barrier.
__device__ __forceinline__ uint64_t ld_dev64(const void* p) {
    return __hip_atomic_load((uint64_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev64(void* p, uint64_t v) {
    __hip_atomic_store((uint64_t*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <bool SC>
__device__ __forceinline__ float2 ld_f2(const float2* p) {
    if (!SC) return *p;
    const uint64_t v = ld_dev64(p);
    return float2{__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32))};
}
template <bool SC>
__device__ __forceinline__ void st_f2(float2* p, float2 v) {
    if (!SC) {
        *p = v;
        return;
    }
    st_dev64(p, (uint64_t)__float_as_uint(v.x) | ((uint64_t)__float_as_uint(v.y) << 32));
}
static_assert(sizeof(RowInfo) == 24, "RowInfo moves as three 64-bit words");
template <bool SC>
__device__ __forceinline__ void st_info(RowInfo* p, const RowInfo& v) {
    if (!SC) {
        *p = v;
        return;
    }
    const uint64_t* w = (const uint64_t*)&v;
    for (int i = 0; i < 3; ++i) st_dev64((uint64_t*)p + i, w[i]);
}
template <bool SC>
__device__ __forceinline__ RowInfo ld_info(const RowInfo* p) {
    if (!SC) return *p;
    RowInfo v;
    uint64_t* w = (uint64_t*)&v;
    for (int i = 0; i < 3; ++i) w[i] = ld_dev64((const uint64_t*)p + i);
    return v;
}

// SC: the statistics are read and the row's RowInfo written device-coherently.
template <int P, bool SC>
__device__ __forceinline__ void row_stats(const MarkovArgs& a, const float2* stats, RowInfo* info, int ntiles,
                                          int k, int r, int lane) {
    const float2* st = stats + (int64_t)r * ntiles;
    const int per = ceil_div(ntiles, DSPARK_WAVE);
    const int t0 = lane * per;
    // the uniform and every tile of the run are loaded up front (clamped
    // indices, then masked: no load waits behind a branch)
    const float uu = a.u[(int64_t)r * a.K + (k - 1)];
    float2 x[P];
#pragma unroll
    for (int i = 0; i < P; ++i) x[i] = ld_f2<SC>(st + min(t0 + i, ntiles - 1));
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int i = 0; i < P; ++i) {
        if (!(i < per && t0 + i < ntiles)) x[i] = float2{-__builtin_huge_valf(), 0.0f};
        m = fmaxf(m, x[i].x);
    }
    const float M = wave_max(m);
    double w[P], loc = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int i = 0; i < P; ++i) {
        w[i] = x[i].x > -__builtin_huge_valf() ? (double)x[i].y * (double)exp2f(x[i].x - M) : 0.0;
        loc += w[i];
        if (w[i] > 0.0) lastpos = t0 + i;
    }
    double incl = loc;  // inclusive prefix over the lanes
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl += t;
    }
    const double total = __shfl(incl, DSPARK_WAVE - 1, DSPARK_WAVE);
    const double thr = (double)uu * total;
    int last = lastpos;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, DSPARK_WAVE));
    // the first lane whose run holds the crossing
    const uint64_t hit = __builtin_amdgcn_ballot_w64(incl > thr && loc > 0.0);
    RowInfo ri;
    ri.M = M;
    ri.S = (float)total;
    ri.pad = 0;
    if (hit != 0) {
        if (lane == __builtin_ctzll(hit)) {
            double cum = incl - loc;
            int pick = -1;
            double before = 0.0;
#pragma unroll
            for (int i = 0; i < P; ++i) {
                if (pick < 0 && w[i] > 0.0 && cum + w[i] > thr) {
                    pick = t0 + i;
                    before = cum;
                }
                cum += w[i];
            }
            if (pick >= 0) {
                ri.tile = pick;
                ri.thr = thr - before;
            } else {  // rounding inside the run: its last tile with mass
                ri.tile = lastpos;
                ri.thr = __builtin_huge_val();
            }
            st_info<SC>(info + r, ri);
        }
    } else if (lane == 0) {
        // rounding pushed u * total past the end: the row's last tile with mass
        ri.tile = max(last, 0);
        ri.thr = __builtin_huge_val();
        st_info<SC>(info + r, ri);
    }
}

template <int P>
__global__ __launch_bounds__(DSPARK_WAVE) void md_stats(MarkovArgs a, const float2* stats, RowInfo* info,
                                                        int ntiles, int k) {
    row_stats<P, false>(a, stats, info, ntiles, k, blockIdx.x, threadIdx.x);
}

inline void stats_pass(const MarkovArgs& a, const float2* stats, RowInfo* info, int ntiles, int k,
                       hipStream_t s) {
    if (ntiles <= DSPARK_WAVE * 16)
        hipLaunchKernelGGL(md_stats<16>, dim3(a.R), dim3(DSPARK_WAVE), 0, s, a, stats, info, ntiles, k);
    else
        hipLaunchKernelGGL(md_stats<kStatsMaxPer>, dim3(a.R), dim3(DSPARK_WAVE), 0, s, a, stats, info, ntiles, k);
}

// ----------------------------------------------------------------- md_norm

// One workgroup per (request, 8192-entry segment of the vocabulary).  The
// request's draft_p row holds z in base-2 units (written by md_tile); it
// becomes p = 2^(z - M) / S in place, every load of the thread issued before
// its first store.  In the workgroup whose segment holds the request's draw
// tile, wave 0 takes that tile's 128 entries itself: their masses 2^(z - M)
// in fp32, the draw (fp64 prefix in vocabulary order; the first entry whose
// running mass passes thr, or the tile's last entry with mass), their p, then
// x_k, and for k < K the next embedding E_next[r] = W1[x_k] and the
// confidence c_{k+1}.  The other threads skip that tile, so nothing else
// writes it.
constexpr int kNormV = 8192;
constexpr int kNormIt = kNormV / (4 * kThreads);  // float4 groups per thread
static_assert(kNormV % kTileV == 0, "a tile lies inside one segment");

template <bool VEC>
__global__ __launch_bounds__(kThreads) void md_norm(MarkovArgs a, const RowInfo* info, uint16_t* E_next,
                                                    const float* sh, int k) {
    const int r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int s0 = blockIdx.y * kNormV;
    const int s1 = min(a.V, s0 + kNormV);
    const int64_t row = (int64_t)r * a.K + (k - 1);
    float* p = a.draft_p + row * a.V;
    const RowInfo ri = info[r];
    const float inv = 1.0f / ri.S;
    const int tb = ri.tile * kTileV;
    const bool draws = tb >= s0 && tb < s1;  // the same in the whole workgroup
    const int skip0 = draws ? tb : s1, skip1 = draws ? tb + kTileV : s1;
    const bool drawer = draws && tid < DSPARK_WAVE;
    float dz[2];
    if (drawer) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int v = tb + 2 * lane + e;
            dz[e] = v < a.V ? p[v] : -__builtin_huge_valf();
        }
    }
    if (VEC) {
        // V % 4 == 0: groups start at multiples of 4, so a group is wholly
        // inside or outside the draw tile and the row
        float4 zv[kNormIt];
#pragma unroll
        for (int i = 0; i < kNormIt; ++i)
            zv[i] = *(const float4*)(p + min(s0 + 4 * (tid + i * kThreads), s1 - 4));
#pragma unroll
        for (int i = 0; i < kNormIt; ++i) {
            const int v = s0 + 4 * (tid + i * kThreads);
            if (v < s1 && (v < skip0 || v >= skip1))
                *(float4*)(p + v) = float4{__builtin_amdgcn_exp2f(zv[i].x - ri.M) * inv,
                                           __builtin_amdgcn_exp2f(zv[i].y - ri.M) * inv,
                                           __builtin_amdgcn_exp2f(zv[i].z - ri.M) * inv,
                                           __builtin_amdgcn_exp2f(zv[i].w - ri.M) * inv};
        }
    } else {
        float zs[4 * kNormIt];
#pragma unroll
        for (int i = 0; i < 4 * kNormIt; ++i) zs[i] = p[min(s0 + tid + i * kThreads, s1 - 1)];
#pragma unroll
        for (int i = 0; i < 4 * kNormIt; ++i) {
            const int v = s0 + tid + i * kThreads;
            if (v < s1 && (v < skip0 || v >= skip1)) p[v] = __builtin_amdgcn_exp2f(zs[i] - ri.M) * inv;
        }
    }
    if (!drawer) return;
    const float q0 = __builtin_amdgcn_exp2f(dz[0] - ri.M), q1 = __builtin_amdgcn_exp2f(dz[1] - ri.M);
    if (tb + 2 * lane < a.V) p[tb + 2 * lane] = q0 * inv;
    if (tb + 2 * lane + 1 < a.V) p[tb + 2 * lane + 1] = q1 * inv;
    const double m0 = q0, m1 = q1;
    double incl = m0 + m1;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl += t;
    }
    const double before = incl - (m0 + m1);  // mass before entry 2 * lane
    // first entry whose running mass passes thr (zero masses are never drawn)
    const int cand = before + m0 > ri.thr && m0 > 0.0 ? 2 * lane
                     : incl > ri.thr && m1 > 0.0    ? 2 * lane + 1
                                                    : kTileV;
    int first = cand;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o, DSPARK_WAVE));
    // rounding: the tile's last entry with mass
    int last = m1 > 0.0 ? 2 * lane + 1 : m0 > 0.0 ? 2 * lane : -1;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, DSPARK_WAVE));
    const int x = tb + (first < kTileV ? first : max(last, 0));
    const bool ok = prev_token(a, r, k) >= 0;
    if (lane == 0) a.draft_tok[row] = ok ? x : -1;
    if (k < a.K) {
        const uint16_t* w1 = a.W1 + (int64_t)(ok ? x : 0) * a.rank;
        for (int q8 = lane * 8; q8 < a.rank; q8 += DSPARK_WAVE * 8)
            *(uint4*)(E_next + (int64_t)r * a.rank + q8) = *(const uint4*)(w1 + q8);
        const float sc = embed_dot(a, w1, lane) + (sh ? sh[row + 1] : 0.0f);
        if (lane == 0) a.conf[row + 1] = ok ? confidence(a, sc, k + 1) : __builtin_nanf("");
    }
}

// One position after the embeddings E are in place: md_tile over every
// vocabulary tile (z and the tile statistics), md_stats, then md_norm, which
// draws x_k and gathers the next embedding into En.
template <int KS, int NT>
void position(const MarkovArgs& a, const uint16_t* E, float2* stats, RowInfo* info, uint16_t* En,
              const float* shp, int ntiles, int k, bool vec, hipStream_t s) {
    const dim3 g(ntiles), b(kThreads);
    if (vec && a.base_bf16) hipLaunchKernelGGL((md_tile<KS, NT, true, true>), g, b, 0, s, a, E, stats, ntiles, k);
    else if (vec) hipLaunchKernelGGL((md_tile<KS, NT, true, false>), g, b, 0, s, a, E, stats, ntiles, k);
    else if (a.base_bf16) hipLaunchKernelGGL((md_tile<KS, NT, false, true>), g, b, 0, s, a, E, stats, ntiles, k);
    else hipLaunchKernelGGL((md_tile<KS, NT, false, false>), g, b, 0, s, a, E, stats, ntiles, k);
    stats_pass(a, stats, info, ntiles, k, s);
    const dim3 gn(a.R, ceil_div(a.V, kNormV));
    if (vec) hipLaunchKernelGGL(md_norm<true>, gn, b, 0, s, a, (const RowInfo*)info, En, shp, k);
    else hipLaunchKernelGGL(md_norm<false>, gn, b, 0, s, a, (const RowInfo*)info, En, shp, k);
}

// ----------------------------------------------------------------- md_coop

// One position of either head (bf16 base logits, V % 4 == 0, at most 1024
// tiles; NT B terms per request: the Markov head's embedding, or the RNN
// head's output as two terms, whose products add up in the accumulators) for
// a group of up to 128 requests in one launch whose workgroups are
// all resident at once (the grid is at most what the device holds, one
// workgroup per CU), with z held in registers from the product to the
// normalisation, so that it never goes through memory: the projection and
// the base logits are read once and p is written once.
//   A  workgroup g owns the tiles g, g + G, g + 2G, g + 3G (G workgroups; 8
//      waves, 16 vocabulary entries of a tile each, the group's requests as 8
//      blocks of 16), so that at each step the grid reads one contiguous
//      stretch of W2t and of every base-logit row: the group's
//      embeddings go to LDS, then per tile z = inv_temp * (U + W2^T e) on
//      v_mfma_f32_16x16x32_bf16, with the next tile's W2t rows and base
//      logits loaded during the current tile's products; z stays in the
//      accumulators (128 AGPRs per lane), and the per-tile statistics (max,
//      sum of 2^(z - max)) go to memory;
//   -  grid barrier;
//   B  one wave per request: row maximum, total and draw tile (the md_stats
//      computation);
//   -  grid barrier;
//   C  the draws of the requests whose draw tile a workgroup owns, eight at
//      a time, one per wave: the tile's masses go through LDS, then the fp64
//      prefix in vocabulary order, x_k, and for k < K the gather of e_{k+1}
//      and c_{k+1}; then every workgroup writes p = 2^(z - M) / S for its
//      tiles from the registers.
// The statistics and row records cross the barriers as device-coherent
// (agent-scope) 64-bit stores and loads, which bypass the per-XCD L2, so the
// barrier needs no L2 write-back or invalidation: a thread's stores are
// complete (s_waitcnt) before its workgroup arrives.  Arrivals are counted per
// group of workgroups (blockIdx % 8) and the last arrival of the last group
// raises every group's flag, which that group's workgroups poll.  Barrier b
// (b = 2L + 1, 2L + 2 for launch L of the block) completes when a group's
// count reaches its size times b; md_first zeroes the counts and flags.
// Residency: the grid never exceeds the workgroups the device holds at once,
// so on an otherwise idle device every workgroup starts at once; if other
// work holds CUs, the missing workgroups start when it ends.  A wait longer
// than kSyncTimeout (2 s) gives up and sets the timeout word, after which
// every barrier of the block returns at once and md_check marks the block's
// outputs invalid (draft tokens -1, confidences NaN): the kernels always
// finish.
constexpr int kCoThreads = 512;
constexpr int kCoWaves = kCoThreads / DSPARK_WAVE;  // 8: 16 entries of a tile each
constexpr int kCoTiles = 4;                         // tiles per workgroup
constexpr int kCoRows = 128;                        // requests per group
constexpr int kCoRT = kCoRows / 16;
constexpr uint64_t kSyncTimeout = 200000000ull;     // wall-clock ticks (100 MHz): 2 s
constexpr int kCoLds = 160 * 1024;                  // LDS of one workgroup (and CU)
static_assert(kCoWaves * 16 == kTileV, "the waves of a workgroup cover one tile");

struct CoopArgs {
    MarkovArgs a;
    const uint16_t* E;  // B operand of position k: row r at E + r * NT * rank (NT bf16 terms)
    uint16_t* E_next;   // embeddings of position k + 1
    float2* stats;      // [R, ntiles]
    RowInfo* info;      // [R]
    const float* sh;    // w_h . h per (r, k), or null
    unsigned* sync;     // kSyncWords barrier words
    int ntiles, k, g0, ng;
    unsigned launch;    // index L of this launch in the block
};

// Keeps a value in accumulation registers (AGPRs) at this point: z lives
// there from the products to the normalisation, leaving the vector registers
// to the loads and the row statistics.
__device__ __forceinline__ void pin_acc(f32x4& v) { asm volatile("" : "+a"(v)); }

__device__ __forceinline__ void grid_barrier(unsigned* sync, unsigned b) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's stores are complete
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned G = gridDim.x, x = blockIdx.x % kCoGroups;
        const unsigned nx = (G - x + kCoGroups - 1) / kCoGroups, ngrp = min(G, (unsigned)kCoGroups);
        if (__hip_atomic_fetch_add(sync + kSyncStride * (1 + x), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) +
                    1u == nx * b &&
            __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u == ngrp * b) {
            for (unsigned y = 0; y < ngrp; ++y)
                __hip_atomic_store(sync + kSyncStride * (1 + kCoGroups + y), b, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
        unsigned* flag = sync + kSyncStride * (1 + kCoGroups + x);
        const uint64_t t0 = wall_clock64();
        while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < b &&
               __hip_atomic_load(sync + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
            __builtin_amdgcn_s_sleep(8);
            if (wall_clock64() - t0 > kSyncTimeout)
                __hip_atomic_store(sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int KS, int NT>
__global__ __launch_bounds__(kCoThreads) void md_coop(CoopArgs c) {
    const MarkovArgs& a = c.a;
    constexpr int kNch = 4 * KS;  // 16-byte chunks per embedding row
    constexpr int kRank = 32 * KS;
    constexpr int kECopy = NT * kCoRows * kNch / kCoThreads;  // embedding chunks per thread
    static_assert(NT * kCoRows * kNch % kCoThreads == 0, "the embedding copy divides evenly");
    // LDS: the group's embeddings (NT terms per request), the per-wave tile
    // statistics, and phase C's draw records, which take the embeddings'
    // place when the three do not fit side by side (the embeddings are no
    // longer read by then)
    constexpr int kSeBytes = NT * kCoRows * kRank * 2;
    constexpr int kSstBytes = kCoTiles * kCoWaves * kCoRows * (int)sizeof(float2);
    constexpr int kInfoBytes = kCoRows * (int)sizeof(RowInfo), kMassBytes = kCoWaves * kTileV * 4;
    constexpr int kDrawBytes = kInfoBytes + kMassBytes + (kCoRows + 4) * 4;
    constexpr bool kShare = kSeBytes + kSstBytes + kDrawBytes > kCoLds;
    static_assert(kSeBytes + kSstBytes <= kCoLds && kDrawBytes <= kSeBytes, "md_coop's LDS fits");
    __shared__ __align__(16) unsigned char smem[kSeBytes + kSstBytes + (kShare ? 0 : kDrawBytes)];
    uint16_t* const se = (uint16_t*)smem;
    float2(*const sst)[kCoWaves][kCoRows] = (float2(*)[kCoWaves][kCoRows])(smem + kSeBytes);
    unsigned char* const sdr = smem + (kShare ? 0 : kSeBytes + kSstBytes);
    RowInfo* const sinfo = (RowInfo*)sdr;
    float(*const smass)[kTileV] = (float(*)[kTileV])(sdr + kInfoBytes);
    int* const sdraw = (int*)(sdr + kInfoBytes + kMassBytes);
    int& ndraw = sdraw[kCoRows];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const int k = c.k, g0 = c.g0;
    // tiles g, g + G, g + 2G, g + 3G: at each step the grid reads one
    // contiguous stretch of every base-logit row and of W2t
    const int Gt = gridDim.x;
    const int nt = min(kCoTiles, (c.ntiles - (int)blockIdx.x + Gt - 1) / Gt);  // >= 1
    auto tile_of = [&](int i) { return (int)blockIdx.x + i * Gt; };
    const unsigned G = gridDim.x;
    const int R = c.ng;
    const int nrt = (R + 15) >> 4;
    constexpr float kLog2e = 1.4426950408889634f;
    const float scale2 = a.inv_temp * kLog2e;

    // A fragments of tile i (W2t rows, clamped into the vocabulary) and its
    // base logits at position k for the group at g0 (entries 4 lq .. 4 lq + 3
    // of this wave's 16, rows 16 rt + lr, 4 bf16 each)
    bf16x8 af[2][KS];
    uint2 ub[2][kCoRT];
    auto load_tile = [&](int i, bf16x8 (&A)[KS], uint2 (&U)[kCoRT]) {
        const int vt = tile_of(i) * kTileV + 16 * wave;
        const uint16_t* src = a.W2t + (int64_t)min(vt + lr, a.V - 1) * kRank + 8 * lq;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) A[ks] = *(const bf16x8*)(src + 32 * ks);
        const int vc = min(vt + 4 * lq, a.V - 4);  // V % 4 == 0
#pragma unroll
        for (int rt = 0; rt < kCoRT; ++rt) {
            const int r = g0 + min(16 * rt + lr, R - 1);
            U[rt] = *(const uint2*)((const uint16_t*)a.base + ((int64_t)r * a.K + (k - 1)) * a.ld + vc);
        }
    };
    // the group's embeddings (rows past the group are zero), then the
    // first tile, which stays in flight past the LDS stores
    uint64_t ev[kECopy][2];
#pragma unroll
    for (int j = 0; j < kECopy; ++j) {
        const int idx = tid + j * kCoThreads, t = idx / (NT * kNch), q = idx % (NT * kNch);
        const uint4 v = *(const uint4*)(c.E + (int64_t)(g0 + min(t, R - 1)) * (NT * kRank) + 8 * q);
        ev[j][0] = t < R ? (uint64_t)v.x | ((uint64_t)v.y << 32) : 0u;
        ev[j][1] = t < R ? (uint64_t)v.z | ((uint64_t)v.w << 32) : 0u;
    }
    load_tile(0, af[0], ub[0]);
#pragma unroll
    for (int j = 0; j < kECopy; ++j) {
        const int idx = tid + j * kCoThreads, t = idx / (NT * kNch), q = idx % (NT * kNch);
        const int nt = q / kNch, ch = q % kNch;
        uint64_t* dst = (uint64_t*)(se + ((nt * kCoRows + t) * kNch + eslot(t, ch, kNch)) * 8);
        dst[0] = ev[j][0];
        dst[1] = ev[j][1];
    }
    lds_barrier();

    // ---- A: products, z in the accumulators, tile statistics
    f32x4 acc[kCoTiles][kCoRT];
#pragma unroll
    for (int i = 0; i < kCoTiles; ++i) {
        if (i + 1 < nt) load_tile(i + 1, af[(i + 1) & 1], ub[(i + 1) & 1]);
#pragma unroll
        for (int rt = 0; rt < kCoRT; ++rt) {
            acc[i][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
            pin_acc(acc[i][rt]);
        }
        if (i < nt) {
#pragma unroll
            for (int rt = 0; rt < kCoRT; ++rt) {
                if (rt < nrt) {
                    const int t = 16 * rt + lr;
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                        for (int ks = 0; ks < KS; ++ks) {
                            const bf16x8 b =
                                *(const bf16x8*)(se + ((nt * kCoRows + t) * kNch + eslot(t, 4 * ks + lq, kNch)) * 8);
                            acc[i][rt] =
                                __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i & 1][ks], b, acc[i][rt], 0, 0, 0);
                        }
                }
            }
            const int vb = tile_of(i) * kTileV + 16 * wave + 4 * lq;
#pragma unroll
            for (int rt = 0; rt < kCoRT; ++rt) {
                const bool ok = vb < a.V && 16 * rt + lr < R;
                const uint2 w = ub[i & 1][rt];
                const float u[4] = {__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                                    __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
                float m = -__builtin_huge_valf();
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float z = ok ? scale2 * (u[e] + acc[i][rt][e]) : -__builtin_huge_valf();
                    acc[i][rt][e] = z;
                    m = fmaxf(m, z);
                }
                m = quad_max(m);
                float s = 0.0f;
                if (m > -__builtin_huge_valf()) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) s += __builtin_amdgcn_exp2f(acc[i][rt][e] - m);
                }
                s = quad_sum(s);
                if (lq == 0) sst[i][wave][16 * rt + lr] = float2{m, s};
                pin_acc(acc[i][rt]);
            }
        }
    }
    lds_barrier();
    {
        const int i = tid / kCoRows, r = tid % kCoRows;  // 512 threads: every (tile, request)
        if (i < nt && r < R) {
            float M = -__builtin_huge_valf();
#pragma unroll
            for (int w = 0; w < kCoWaves; ++w) M = fmaxf(M, sst[i][w][r].x);
            float S = 0.0f;
            if (M > -__builtin_huge_valf()) {
#pragma unroll
                for (int w = 0; w < kCoWaves; ++w)
                    if (sst[i][w][r].x > -__builtin_huge_valf())
                        S += sst[i][w][r].y * exp2f(sst[i][w][r].x - M);
            }
            st_f2<true>(c.stats + (int64_t)(g0 + r) * c.ntiles + tile_of(i), float2{M, S});
        }
    }
    grid_barrier(c.sync, 2u * c.launch + 1u);

    // ---- B: row statistics, one wave per request
    for (int r = blockIdx.x + (int)G * wave; r < R; r += (int)G * kCoWaves)
        row_stats<16, true>(a, c.stats, c.info, c.ntiles, k, g0 + r, lane);
    grid_barrier(c.sync, 2u * c.launch + 2u);
#pragma unroll
    for (int i = 0; i < kCoTiles; ++i)
#pragma unroll
        for (int rt = 0; rt < kCoRT; ++rt) pin_acc(acc[i][rt]);

    // ---- C: the draws of the tiles owned here, then p from the registers
    // (the draws first: a load waits for every store issued before it, and
    // the draw's gathers would queue behind the p stores)
    if (tid == 0) ndraw = 0;
    if (tid < R) sinfo[tid] = ld_info<true>(c.info + g0 + tid);
    lds_barrier();
    if (tid < R) {
        const int d = sinfo[tid].tile - (int)blockIdx.x;
        if (d >= 0 && d % Gt == 0 && d / Gt < nt) sdraw[atomicAdd(&ndraw, 1)] = tid;
    }
    lds_barrier();  // the draw list is complete
    const int nd = ndraw;
    for (int j0 = 0; j0 < nd; j0 += kCoWaves) {
        // every wave puts its 16 entries of each draw tile of this round into LDS
        for (int j = j0; j < min(nd, j0 + kCoWaves); ++j) {
            const int rl = sdraw[j];
            const int ti = (sinfo[rl].tile - (int)blockIdx.x) / Gt;
            const float M = sinfo[rl].M;
#pragma unroll
            for (int i = 0; i < kCoTiles; ++i)
#pragma unroll
                for (int rt = 0; rt < kCoRT; ++rt)
                    if (i == ti && 16 * rt + lr == rl) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            smass[j - j0][16 * wave + 4 * lq + e] = __builtin_amdgcn_exp2f(acc[i][rt][e] - M);
                    }
        }
        lds_barrier();
        if (j0 + wave < nd) {  // wave w makes draw j0 + w
            const int rl = sdraw[j0 + wave];
            const RowInfo ri = sinfo[rl];
            const int r = g0 + rl;
            const int64_t row = (int64_t)r * a.K + (k - 1);
            const double m0 = smass[wave][2 * lane], m1 = smass[wave][2 * lane + 1];
            double incl = m0 + m1;
#pragma unroll
            for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
                const double t = __shfl_up(incl, o, DSPARK_WAVE);
                if (lane >= o) incl += t;
            }
            const double before = incl - (m0 + m1);  // mass before entry 2 * lane
            // first entry whose running mass passes thr (zero masses are never drawn)
            const int cand = before + m0 > ri.thr && m0 > 0.0 ? 2 * lane
                             : incl > ri.thr && m1 > 0.0    ? 2 * lane + 1
                                                            : kTileV;
            int first = cand;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o, DSPARK_WAVE));
            // rounding: the tile's last entry with mass
            int last = m1 > 0.0 ? 2 * lane + 1 : m0 > 0.0 ? 2 * lane : -1;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, DSPARK_WAVE));
            const int x = ri.tile * kTileV + (first < kTileV ? first : max(last, 0));
            const bool ok = prev_token(a, r, k) >= 0;
            if (lane == 0) a.draft_tok[row] = ok ? x : -1;
            if (k < a.K) {
                const uint16_t* w1 = a.W1 + (int64_t)(ok ? x : 0) * a.rank;
                for (int q8 = lane * 8; q8 < a.rank; q8 += DSPARK_WAVE * 8)
                    *(uint4*)(c.E_next + (int64_t)r * a.rank + q8) = *(const uint4*)(w1 + q8);
                const float sc = embed_dot(a, w1, lane) + (c.sh ? c.sh[row + 1] : 0.0f);
                if (lane == 0) a.conf[row + 1] = ok ? confidence(a, sc, k + 1) : __builtin_nanf("");
            }
        }
        // (after the last round the other waves go on to the p stores)
        if (j0 + kCoWaves < nd) lds_barrier();
    }
    float rm[kCoRT], rinv[kCoRT];
#pragma unroll
    for (int rt = 0; rt < kCoRT; ++rt) {
        const RowInfo ri = sinfo[min(16 * rt + lr, R - 1)];
        rm[rt] = ri.M;
        rinv[rt] = 1.0f / ri.S;
    }
#pragma unroll
    for (int i = 0; i < kCoTiles; ++i) {
        const int vb = tile_of(i) * kTileV + 16 * wave + 4 * lq;
        if (i < nt && vb < a.V) {
#pragma unroll
            for (int rt = 0; rt < kCoRT; ++rt) {
                const int r = 16 * rt + lr;
                if (r < R) {
                    float* out = a.draft_p + ((int64_t)(g0 + r) * a.K + (k - 1)) * a.V + vb;
                    *(float4*)out = float4{__builtin_amdgcn_exp2f(acc[i][rt][0] - rm[rt]) * rinv[rt],
                                           __builtin_amdgcn_exp2f(acc[i][rt][1] - rm[rt]) * rinv[rt],
                                           __builtin_amdgcn_exp2f(acc[i][rt][2] - rm[rt]) * rinv[rt],
                                           __builtin_amdgcn_exp2f(acc[i][rt][3] - rm[rt]) * rinv[rt]};
                }
            }
        }
    }
}

// After the block's md_coop launches: when one of their barriers gave up
// waiting, no output of the block is valid (draft tokens -1, confidences NaN).
__global__ __launch_bounds__(kThreads) void md_check(MarkovArgs a, const unsigned* sync) {
    if (sync[1] == 0u) return;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < (int64_t)a.R * a.K) {
        a.draft_tok[i] = -1;
        a.conf[i] = __builtin_nanf("");
    }
}

// Workgroups of md_coop<KS, NT> that the current device holds at once (0 when
// it cannot tell); computed once per device.
template <int KS, int NT>
int coop_grid_limit() {
    constexpr int kMaxDevices = 64;
    static int cache[kMaxDevices];  // 0: not yet asked, -1: none
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
    if (cache[dev] == 0) {
        int cus = 0, nb = 0;
        const bool ok = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, md_coop<KS, NT>, kCoThreads, 0) == hipSuccess;
        cache[dev] = ok && nb * cus > 0 ? nb * cus : -1;
    }
    return cache[dev] > 0 ? cache[dev] : 0;
}

// One position as md_coop launches, one per group of up to 128 requests
// (launch counts the block's launches: it numbers their barriers).
template <int KS, int NT>
void coop_position(const MarkovArgs& a, const uint16_t* E, uint16_t* En, float2* stats, RowInfo* info,
                   const float* shp, unsigned* sync, int ntiles, int k, unsigned& launch, hipStream_t s) {
    const int G = ceil_div(ntiles, kCoTiles);
    for (int g0 = 0; g0 < a.R; g0 += kCoRows) {
        CoopArgs c;
        c.a = a;
        c.E = E;
        c.E_next = En;
        c.stats = stats;
        c.info = info;
        c.sh = shp;
        c.sync = sync;
        c.ntiles = ntiles;
        c.k = k;
        c.g0 = g0;
        c.ng = std::min(kCoRows, a.R - g0);
        c.launch = launch++;
        hipLaunchKernelGGL((md_coop<KS, NT>), dim3(G), dim3(kCoThreads), 0, s, c);
    }
}

// md_coop applies: bf16 base logits, V % 4 == 0 (vec), at most 1024 tiles
// (the row statistics' 16 tiles per lane), and a grid the device holds at once.
template <int KS, int NT>
bool coop_applies(const MarkovArgs& a, int ntiles, bool vec) {
    return vec && a.base_bf16 && ntiles <= DSPARK_WAVE * 16 &&
           ceil_div(ntiles, kCoTiles) <= coop_grid_limit<KS, NT>();
}

// ------------------------------------------------------------ RNN head

// The backbone part of the RNN head's projection (eq. rnn), once for every
// (request, position) since it does not depend on the drawn tokens:
// Hp[row, i] = sum_{j < d} Wrnn[i, 2 rank + j] h[row, j], row = r K + k - 1,
// i < 3 rank.  v_mfma_f32_16x16x32_bf16; a workgroup computes 64 rows x 128
// outputs.  Wave w owns rows 16 w .. 16 w + 15 and reads its hidden-state
// fragments straight from memory, one step ahead; the 128 weight rows of each
// 32-input step are staged once per workgroup in an LDS double buffer (row
// pitch 80 bytes) and shared by the four waves.  d % 8 == 0, so a lane's 8
// inputs are either all inside the row or all past its end.
constexpr int kHpRows = 64, kHpCols = 128, kHpNt = kHpCols / 16, kHpPitch = 40;
__global__ __launch_bounds__(kThreads) void rnn_hproj(MarkovArgs a, float* Hp) {
    __shared__ __align__(16) uint16_t sb[2][kHpCols * kHpPitch];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lq = lane >> 4;
    const int nrows = a.R * a.K, ncols = 3 * a.rank, nz = 2 * a.rank + a.d;
    const int m0 = blockIdx.x * kHpRows + 16 * wave;
    const int n0 = blockIdx.y * kHpCols;
    // row starts (hidden row; a weight row's hidden columns): a lane's 8 inputs
    // past the end of the row read the row's first 8 instead (always inside the
    // row, d >= 8) and are zeroed
    const uint16_t* arow = a.hidden + (int64_t)min(m0 + lr, nrows - 1) * a.d;
    // this thread's two 16-byte pieces of a step's weight tile: piece c is row
    // c / 4, input chunk c % 4
    const uint16_t* brow[2];
    int bdst[2], bpart[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int c = tid + kThreads * i;
        bpart[i] = c & 3;
        brow[i] = a.Wrnn + (int64_t)min(n0 + (c >> 2), ncols - 1) * nz + 2 * a.rank;
        bdst[i] = (c >> 2) * kHpPitch + 8 * bpart[i];
    }
    const int nsteps = ceil_div(a.d, 32);
    auto load_a = [&](int st) {
        const int kk = 32 * st + 8 * lq;
        const bool in = st < nsteps && kk < a.d;
        const bf16x8 v = *(const bf16x8*)(arow + (in ? kk : 0));
        return in ? v : bf16x8{};
    };
    auto load_b = [&](int st, uint4* v) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int kk = 32 * st + 8 * bpart[i];
            const bool in = st < nsteps && kk < a.d;
            const uint4 w = *(const uint4*)(brow[i] + (in ? kk : 0));
            v[i] = in ? w : uint4{0u, 0u, 0u, 0u};
        }
    };
    f32x4 acc[kHpNt];
#pragma unroll
    for (int nt = 0; nt < kHpNt; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 vb[2];
    load_b(0, vb);
    bf16x8 a_cur = load_a(0), a_next = load_a(1);
#pragma unroll
    for (int i = 0; i < 2; ++i) *(uint4*)(&sb[0][bdst[i]]) = vb[i];
    __syncthreads();
    for (int st = 0; st < nsteps; ++st) {
        load_b(st + 1, vb);  // the next step's tile stays in flight during the products
        const uint16_t* cur = sb[st & 1];
#pragma unroll
        for (int nt = 0; nt < kHpNt; ++nt) {
            const bf16x8 bfrag = *(const bf16x8*)(cur + (16 * nt + lr) * kHpPitch + 8 * lq);
            acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_cur, bfrag, acc[nt], 0, 0, 0);
        }
        a_cur = a_next;
        a_next = load_a(st + 2);
        // the other buffer was last read in step st - 1, before the barrier that ended it
#pragma unroll
        for (int i = 0; i < 2; ++i) *(uint4*)(&sb[(st + 1) & 1][bdst[i]]) = vb[i];
        __syncthreads();
    }
    // lane holds rows m0 + 4 lq + e, output n0 + 16 nt + lr
#pragma unroll
    for (int nt = 0; nt < kHpNt; ++nt) {
        const int col = n0 + 16 * nt + lr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = m0 + 4 * lq + e;
            if (row < nrows && col < ncols) Hp[(int64_t)row * ncols + col] = acc[nt][e];
        }
    }
}

// hi + mid (+ lo): each term the bf16 rounding of what the previous ones
// leave; hi + mid is v to within 2^-16 |v|, hi + mid + lo to fp32 accuracy
__device__ __forceinline__ void split2(float v, uint16_t* dst, int stride) {
    const uint16_t hi = f32_to_bf16(v);
    dst[0] = hi;
    dst[stride] = f32_to_bf16(v - bf16_to_f32(hi));
}
__device__ __forceinline__ void split3(float v, uint16_t* dst, int stride) {
    const uint16_t hi = f32_to_bf16(v);
    const float r1 = v - bf16_to_f32(hi);
    const uint16_t mid = f32_to_bf16(r1);
    dst[0] = hi;
    dst[stride] = mid;
    dst[2 * stride] = f32_to_bf16(r1 - bf16_to_f32(mid));
}

// Position k of the RNN head on the matrix cores: a = Hp[r, k] + Wrnn[:, :2 rank]
// [s_{k-1}; e_k], e_k = W1[x_{k-1}] gathered by the previous position's draw.
// The K dimension runs over 4 rank inputs: the fp32 state as three bf16 terms
// (hi, mid, lo; written by the previous position) against the state columns
// three times, then the exact bf16 embedding against the embedding columns.
// The output columns of a workgroup are the gate, candidate and output rows of
// 16 state dims, so a lane holds all three pre-activations of one (request,
// dim) and applies the gated update in registers: s_k = g s_{k-1} + (1 - g)
// tanh(a_c) with g = sigmoid(a_g), written in fp32 and as three terms, and the
// head's output o_k = tanh(a_o) as two terms (hi, mid) for the vocabulary
// product.  A workgroup owns
// 16 dims x 16 requests; its four waves take every fourth 32-input step (both
// operands straight from memory, kStDepth steps ahead) and wave 0 adds the
// four partial products in wave order.  The state is double-buffered (others
// may still read s_{k-1}); at k = 1 it is zero and its steps are skipped.
constexpr int kStJ = 16, kStR = 16, kStDepth = 4;
__global__ __launch_bounds__(kThreads) void rnn_state(MarkovArgs a, const float* Hp,
                                                      const float* s_prev, const uint16_t* S3_prev,
                                                      float* s_next, uint16_t* S3_next,
                                                      const uint16_t* Ee, uint16_t* E2, int k) {
    __shared__ f32x4 part[kWaves - 1][3][DSPARK_WAVE];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, lq = lane >> 4;
    const int rank = a.rank, nz = 2 * rank + a.d;
    const int j0 = blockIdx.x * kStJ;
    const int m0 = blockIdx.y * kStR;
    const int ra = min(m0 + lr, a.R - 1);  // request of this lane's A fragment
    const int ks_s = 3 * rank / 32, nst = ks_s + rank / 32;
    const int st0 = (k > 1 ? 0 : ks_s) + wave;  // this wave's steps: st0, st0 + 4, ...
    bf16x8 af[kStDepth], bfr[kStDepth][3];
    auto load = [&](int i, int slot) {  // this wave's i-th step
        const int kk = 32 * min(st0 + kWaves * i, nst - 1) + 8 * lq;  // past the end: unused
        const bool state = kk < 3 * rank;                            // uniform over the wave
        af[slot] = state ? *(const bf16x8*)(S3_prev + (int64_t)ra * 3 * rank + kk)
                         : *(const bf16x8*)(Ee + (int64_t)ra * rank + (kk - 3 * rank));
        const int col = state ? kk % rank : kk - 2 * rank;
#pragma unroll
        for (int p = 0; p < 3; ++p)
            bfr[slot][p] = *(const bf16x8*)(a.Wrnn + (int64_t)(p * rank + j0 + lr) * nz + col);
    };
    const int nmine = st0 < nst ? (nst - st0 + kWaves - 1) / kWaves : 0;
    // wave 0's epilogue inputs (the projection of the hidden states and the
    // previous state of its requests m0 + 4 lq + e, dim j0 + lr) do not depend
    // on the products: they are loaded first (rows clamped, then masked)
    const int j = j0 + lr;
    float hpv[4][3], spv[4];
    if (wave == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rc = min(m0 + 4 * lq + e, a.R - 1);
            const float* hp = Hp ? Hp + ((int64_t)rc * a.K + (k - 1)) * (3 * rank) : nullptr;
#pragma unroll
            for (int p = 0; p < 3; ++p) hpv[e][p] = hp ? hp[p * rank + j] : 0.0f;
            spv[e] = k > 1 ? s_prev[(int64_t)rc * rank + j] : 0.0f;
        }
    }
    f32x4 acc[3];
#pragma unroll
    for (int p = 0; p < 3; ++p) acc[p] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kStDepth; ++u) load(u, u);
    for (int i0 = 0; i0 < nmine; i0 += kStDepth) {
#pragma unroll
        for (int u = 0; u < kStDepth; ++u) {
            if (i0 + u < nmine) {
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u], bfr[u][p], acc[p], 0, 0, 0);
            }
            load(i0 + kStDepth + u, u);
        }
    }
    if (wave > 0) {
#pragma unroll
        for (int p = 0; p < 3; ++p) part[wave - 1][p][lane] = acc[p];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 0; w < kWaves - 1; ++w)
#pragma unroll
        for (int p = 0; p < 3; ++p) acc[p] += part[w][p][lane];
    // lane holds requests m0 + 4 lq + e, state dim j0 + lr
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int r = m0 + 4 * lq + e;
        if (r >= a.R) continue;
        float ag = acc[0][e], ac = acc[1][e], ao = acc[2][e];
        if (Hp) {
            ag += hpv[e][0];
            ac += hpv[e][1];
            ao += hpv[e][2];
        }
        const float g = 1.0f / (1.0f + expf(-ag));
        const float sp = spv[e];
        const float sn = g * sp + (1.0f - g) * tanhf(ac);
        s_next[(int64_t)r * rank + j] = sn;
        split3(sn, S3_next + (int64_t)r * 3 * rank + j, rank);
        split2(tanhf(ao), E2 + (int64_t)r * 2 * rank + j, rank);
    }
}

template <int KS>
hipError_t launch_rnn_ks(const MarkovArgs& a, uint16_t* Ee, uint16_t* E2, float* S0, float* S1,
                         uint16_t* T0, uint16_t* T1, float* Hp, float2* stats, RowInfo* info,
                         float* sh, unsigned* sync, int ntiles, bool vec, hipStream_t s) {
    const int64_t rows = (int64_t)a.R * a.K;
    if (a.d > 0) {
        hipLaunchKernelGGL(md_hidden, dim3((unsigned)ceil_div((int)rows, kWaves)), dim3(kThreads), 0, s, a, sh);
        hipLaunchKernelGGL(rnn_hproj, dim3((unsigned)ceil_div((int)rows, kHpRows), ceil_div(3 * a.rank, kHpCols)),
                           dim3(kThreads), 0, s, a, Hp);
    }
    const float* shp = a.d > 0 ? sh : nullptr;
    const float* hpp = a.d > 0 ? Hp : nullptr;
    hipLaunchKernelGGL(md_first, dim3(ceil_div(a.R, kWaves)), dim3(kThreads), 0, s, a, shp, Ee, sync);
    // the vocabulary product with the output's two terms: md_coop where it
    // applies, else md_tile, md_stats and md_norm
    const bool coop = coop_applies<KS, 2>(a, ntiles, vec);
    unsigned launch = 0;
    for (int k = 1; k <= a.K; ++k) {
        // s_{k-1} in fp32 and as three terms (unread at k = 1), and where s_k goes
        const float* sp = (k & 1) ? S1 : S0;
        float* sn = (k & 1) ? S0 : S1;
        const uint16_t* tp = (k & 1) ? T1 : T0;
        uint16_t* tn = (k & 1) ? T0 : T1;
        hipLaunchKernelGGL(rnn_state, dim3(a.rank / kStJ, ceil_div(a.R, kStR)), dim3(kThreads), 0, s, a, hpp,
                           sp, tp, sn, tn, (const uint16_t*)Ee, E2, k);
        // the draw gathers W1[x_k] into Ee: the embedding input of position k + 1
        if (coop) coop_position<KS, 2>(a, E2, Ee, stats, info, shp, sync, ntiles, k, launch, s);
        else position<KS, 2>(a, E2, stats, info, Ee, shp, ntiles, k, vec, s);
    }
    if (coop)
        hipLaunchKernelGGL(md_check, dim3((unsigned)ceil_div((int)rows, kThreads)), dim3(kThreads), 0, s, a,
                           (const unsigned*)sync);
    return hipGetLastError();
}

template <int KS>
hipError_t launch_ks(const MarkovArgs& a, uint16_t* E0, uint16_t* E1, float2* stats, RowInfo* info,
                     float* sh, unsigned* sync, int ntiles, bool vec, hipStream_t s) {
    const int64_t rows = (int64_t)a.R * a.K;
    if (a.d > 0) hipLaunchKernelGGL(md_hidden, dim3((unsigned)ceil_div((int)rows, kWaves)), dim3(kThreads), 0, s, a, sh);
    const float* shp = a.d > 0 ? sh : nullptr;
    hipLaunchKernelGGL(md_first, dim3(ceil_div(a.R, kWaves)), dim3(kThreads), 0, s, a, shp, E0, sync);
    // one md_coop launch per position and group of 128 requests where it
    // applies; three launches per position otherwise
    const bool coop = coop_applies<KS, 1>(a, ntiles, vec);
    unsigned launch = 0;
    for (int k = 1; k <= a.K; ++k) {
        uint16_t* Ek = (k & 1) ? E0 : E1;
        uint16_t* En = (k & 1) ? E1 : E0;
        if (coop) coop_position<KS, 1>(a, Ek, En, stats, info, shp, sync, ntiles, k, launch, s);
        else position<KS, 1>(a, Ek, stats, info, En, shp, ntiles, k, vec, s);
    }
    if (coop)
        hipLaunchKernelGGL(md_check, dim3((unsigned)ceil_div((int)rows, kThreads)), dim3(kThreads), 0, s, a,
                           (const unsigned*)sync);
    return hipGetLastError();
}

}  // namespace mkd

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

namespace {
struct WsLayout {
    size_t e, stats, info, sh, sync, total;
};
WsLayout ws_layout(int R, int K, int V, int rank) {
    const int ntiles = mkd::ceil_div(V, mkd::kTileV);
    WsLayout l;
    l.e = align256((size_t)R * rank * 2);
    l.stats = align256((size_t)R * ntiles * sizeof(float2));
    l.info = align256((size_t)R * sizeof(mkd::RowInfo));
    l.sh = align256((size_t)R * K * sizeof(float));
    l.sync = align256(mkd::kSyncWords * sizeof(unsigned));  // md_coop's barrier words
    l.total = 2 * l.e + l.stats + l.info + l.sh + l.sync;
    return l;
}
}  // namespace

size_t markov_workspace(int R, int K, int V, int rank) { return ws_layout(R, K, V, rank).total; }

namespace {
// RNN head: the embedding input Ee, the two-term output E2, two state
// buffers (fp32 and three terms), the backbone part of the projection, then
// what the Markov head uses
struct RnnLayout {
    size_t ee, e2, st, st3, hp, stats, info, sh, sync, total;
};
RnnLayout rnn_layout(int R, int K, int V, int rank) {
    const int ntiles = mkd::ceil_div(V, mkd::kTileV);
    RnnLayout l;
    l.ee = align256((size_t)R * rank * 2);
    l.e2 = align256((size_t)R * 2 * rank * 2);
    l.st = align256((size_t)R * rank * 4);
    l.st3 = align256((size_t)R * 3 * rank * 2);
    l.hp = align256((size_t)R * K * 3 * rank * 4);
    l.stats = align256((size_t)R * ntiles * sizeof(float2));
    l.info = align256((size_t)R * sizeof(mkd::RowInfo));
    l.sh = align256((size_t)R * K * sizeof(float));
    l.sync = align256(mkd::kSyncWords * sizeof(unsigned));
    l.total = l.ee + l.e2 + 2 * l.st + 2 * l.st3 + l.hp + l.stats + l.info + l.sh + l.sync;
    return l;
}
}  // namespace

size_t rnn_workspace(int R, int K, int V, int rank) { return rnn_layout(R, K, V, rank).total; }

hipError_t launch_rnn(const MarkovArgs& a, void* ws, hipStream_t s) {
    const int ntiles = mkd::ceil_div(a.V, mkd::kTileV);
    const RnnLayout l = rnn_layout(a.R, a.K, a.V, a.rank);
    char* p = (char*)ws;
    uint16_t* Ee = (uint16_t*)p;                 p += l.ee;
    uint16_t* E2 = (uint16_t*)p;                 p += l.e2;
    float* S0 = (float*)p;                       p += l.st;
    float* S1 = (float*)p;                       p += l.st;
    uint16_t* T0 = (uint16_t*)p;                 p += l.st3;
    uint16_t* T1 = (uint16_t*)p;                 p += l.st3;
    float* Hp = (float*)p;                       p += l.hp;
    float2* stats = (float2*)p;                  p += l.stats;
    mkd::RowInfo* info = (mkd::RowInfo*)p;       p += l.info;
    float* sh = (float*)p;                       p += l.sh;
    unsigned* sync = (unsigned*)p;
    const size_t eb = a.base_bf16 ? 2 : 4;
    const bool vec = a.V % 4 == 0 && a.ld % 4 == 0 && ((uintptr_t)a.base % (4 * eb)) == 0 &&
                     ((uintptr_t)a.draft_p % 16) == 0;
    switch (a.rank) {
        case 32: return mkd::launch_rnn_ks<1>(a, Ee, E2, S0, S1, T0, T1, Hp, stats, info, sh, sync, ntiles, vec, s);
        case 64: return mkd::launch_rnn_ks<2>(a, Ee, E2, S0, S1, T0, T1, Hp, stats, info, sh, sync, ntiles, vec, s);
        case 128: return mkd::launch_rnn_ks<4>(a, Ee, E2, S0, S1, T0, T1, Hp, stats, info, sh, sync, ntiles, vec, s);
        default: return mkd::launch_rnn_ks<8>(a, Ee, E2, S0, S1, T0, T1, Hp, stats, info, sh, sync, ntiles, vec, s);
    }
}

bool markov_rank_supported(int rank) { return rank == 32 || rank == 64 || rank == 128 || rank == 256; }

int markov_max_vocab() { return DSPARK_WAVE * mkd::kStatsMaxPer * mkd::kTileV; }

hipError_t launch_markov(const MarkovArgs& a, void* ws, hipStream_t s) {
    const int ntiles = mkd::ceil_div(a.V, mkd::kTileV);
    const WsLayout l = ws_layout(a.R, a.K, a.V, a.rank);
    char* p = (char*)ws;
    uint16_t* E0 = (uint16_t*)p;
    uint16_t* E1 = (uint16_t*)(p + l.e);
    float2* stats = (float2*)(p + 2 * l.e);
    mkd::RowInfo* info = (mkd::RowInfo*)(p + 2 * l.e + l.stats);
    float* sh = (float*)(p + 2 * l.e + l.stats + l.info);
    unsigned* sync = (unsigned*)(p + 2 * l.e + l.stats + l.info + l.sh);
    const size_t eb = a.base_bf16 ? 2 : 4;
    const bool vec = a.V % 4 == 0 && a.ld % 4 == 0 && ((uintptr_t)a.base % (4 * eb)) == 0 &&
                     ((uintptr_t)a.draft_p % 16) == 0;
    switch (a.rank) {
        case 32: return mkd::launch_ks<1>(a, E0, E1, stats, info, sh, sync, ntiles, vec, s);
        case 64: return mkd::launch_ks<2>(a, E0, E1, stats, info, sh, sync, ntiles, vec, s);
        case 128: return mkd::launch_ks<4>(a, E0, E1, stats, info, sh, sync, ntiles, vec, s);
        default: return mkd::launch_ks<8>(a, E0, E1, stats, info, sh, sync, ntiles, vec, s);
    }
}

}  // namespace dspark

// Ragged causal verify attention, bf16, head dim 128, on gfx950 matrix cores.
//
// Work item = (request r, KV head g, KV split s, row chunk rc).  The rows of an
// item are the request's q_len verify tokens times the GQA group, packed
// row = t * group + head_in_group, up to 64 per chunk (four 16-row tiles).
// A split covers about 2048 keys; the workgroup's four waves each stream a
// contiguous quarter of it in 32-key steps:
//   S^T[key, row] = K Q^T      v_mfma_f32_16x16x32_bf16, K rows loaded straight
//                              from the page into the A operand (16-byte loads);
//   online softmax per row     exp2 on log2e-scaled scores, causal and length
//                              masks, P rounded to bf16;
//   O^T[d, row] += V^T P^T     V staged through LDS and read transposed as the
//                              A operand; P^T is already in B-operand layout.
// The key order inside a 32-key step is permuted so that the score tile's
// accumulator layout equals the B-operand layout of the second product (no
// shuffles).  The waves are combined through LDS in a fixed order; splits are
// combined by the last workgroup of an item to finish (fixed split order), so
// results are reproducible bit for bit.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace dspark {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kMfThreads = 256;
constexpr int kMfWaves = 4;
constexpr int kSplit = 2048;   // keys per split (upper bound)
constexpr int kStep = 32;      // keys per inner step
constexpr int kNT = 4;         // 16-row tiles per item
constexpr int kRows = 16 * kNT;
constexpr int kD = 128;
constexpr int kVPitch = 264;   // bytes per staged V row (256 + 8: conflict-free column reads)
constexpr int kOPitch = 68;    // floats per d row of the wave-merge buffer
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kSlotFloats = kRows * (kD + 2);

bool attn_mfma_supported(const AttnArgs& a) {
    return a.bf16 && a.Dqk == kD && a.Dv == kD && a.page % kStep == 0 && a.Hq % a.Hkv == 0 &&
           a.ks[2] % 8 == 0 && a.vs[2] % 8 == 0 && a.ks[1] % 8 == 0 && a.vs[1] % 8 == 0 &&
           a.ks[0] % 8 == 0 && a.vs[0] % 8 == 0 && ((uintptr_t)a.q % 16) == 0 &&
           ((uintptr_t)a.k % 16) == 0 && ((uintptr_t)a.v % 16) == 0;
}

struct MfGeom {
    int group, max_splits, rc_max;
    int64_t n_items;
    size_t counter_bytes, part_bytes;
};

static MfGeom mf_geom(const AttnArgs& a) {
    MfGeom g;
    g.group = a.Hq / a.Hkv;
    const int64_t max_kv = (int64_t)a.max_pages * a.page;
    g.max_splits = (int)std::max<int64_t>(1, (max_kv + kSplit - 1) / kSplit);
    g.rc_max = (a.max_q * g.group + kRows - 1) / kRows;
    g.n_items = (int64_t)a.R * a.Hkv * g.max_splits;
    const int64_t slots = (int64_t)a.R * a.Hkv * g.rc_max;
    g.counter_bytes = ((size_t)slots * sizeof(int) + 255) & ~(size_t)255;
    g.part_bytes = (size_t)slots * g.max_splits * kSlotFloats * sizeof(float);
    return g;
}

size_t attn_mfma_workspace(const AttnArgs& a) {
    const MfGeom g = mf_geom(a);
    return g.counter_bytes + g.part_bytes;
}

struct MfParams {
    AttnArgs a;
    int group, max_splits, rc_max;
    int64_t n_items;
    float scale2;
    int* counters;
    float* part;
};

__global__ void mf_zero(int* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__global__ __launch_bounds__(kMfThreads) void attn_mfma_kernel(MfParams p) {
    const AttnArgs& a = p.a;
    // LDS: per-wave staged V (4 x 32 x 264 B) / later the wave-merge buffer (128 x 68 floats)
    __shared__ __align__(16) unsigned char lds[kD * kOPitch * 4];
    __shared__ float s_m[kMfWaves][kRows];
    __shared__ float s_l[kMfWaves][kRows];
    __shared__ int s_last;

    // ---- item decode: consecutive items go to different XCDs, the row chunks of
    // one item share an XCD (blockIdx % 8 selects the XCD)
    const int b = blockIdx.x;
    const int xcd = b & 7;
    const int y = b >> 3;
    const int rc = y % p.rc_max;
    const int64_t item = (int64_t)(y / p.rc_max) * 8 + xcd;
    if (item >= p.n_items) return;
    const int s = (int)(item % p.max_splits);
    const int rg = (int)(item / p.max_splits);
    const int g = rg % a.Hkv;
    const int r = rg / a.Hkv;
    const int q0 = a.cu_q[r];
    const int ql = a.cu_q[r + 1] - q0;
    const int kv = a.kv_len[r];
    if (ql < 1 || ql > a.max_q || kv < ql || kv > a.max_pages * a.page) return;
    const int rows = ql * p.group;
    const int row0 = rc * kRows;
    if (row0 >= rows) return;
    const int nsplit = (kv + kSplit - 1) / kSplit;
    if (s >= nsplit) return;
    const int start = (int)(((int64_t)s * kv / nsplit) & ~(int64_t)(kStep - 1));
    const int end = (s + 1 == nsplit) ? kv
                                      : (int)(((int64_t)(s + 1) * kv / nsplit) & ~(int64_t)(kStep - 1));
    const int nrows = min(kRows, rows - row0);
    const int nt = (nrows + 15) >> 4;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lr = lane & 15;
    const int lq = lane >> 4;

    const uint16_t* __restrict__ qg = (const uint16_t*)a.q;
    const uint16_t* __restrict__ kc = (const uint16_t*)a.k;
    const uint16_t* __restrict__ vc = (const uint16_t*)a.v;
    const int32_t* __restrict__ bt = a.block_table + (int64_t)r * a.max_pages;

    // ---- query fragments (B operand of S^T = K Q^T) and causal limits
    bf16x8 qf[kNT][4];
    int lim[kNT];
#pragma unroll
    for (int i = 0; i < kNT; ++i) {
        const int row = row0 + 16 * i + lr;
        if (row < rows) {
            const int t = row / p.group;
            const int h = g * p.group + (row - t * p.group);
            const uint16_t* qp = qg + ((int64_t)(q0 + t) * a.Hq + h) * kD + 8 * lq;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) qf[i][ks] = *(const bf16x8*)(qp + 32 * ks);
            lim[i] = kv - ql + t;
        } else {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) qf[i][ks] = bf16x8{};
            lim[i] = -1;
        }
    }

    f32x4 acc[kNT][8];
    float mrow[kNT], lsum[kNT];
#pragma unroll
    for (int i = 0; i < kNT; ++i) {
        mrow[i] = -__builtin_huge_valf();
        lsum[i] = 0.0f;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[i][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    const int nblk = (end - start + kStep - 1) / kStep;
    const int b0 = wave * nblk / kMfWaves;
    const int b1 = (wave + 1) * nblk / kMfWaves;
    unsigned char* vt = lds + wave * kStep * kVPitch;

    // key held by this lane as the A-operand row of the score product, per 16-key half
    const int tau0 = 8 * (lr >> 2) + (lr & 3);

    bf16x8 kf[2][4];
    uint4 vr[8];
    auto load_step = [&](int blk) {
        const int tok0 = start + blk * kStep;
        const int64_t page = bt[tok0 / a.page];
        const int slot0 = tok0 % a.page;
        const uint16_t* kb = kc + page * a.ks[0] + (int64_t)g * a.ks[1] + (int64_t)slot0 * a.ks[2];
        const uint16_t* vb = vc + page * a.vs[0] + (int64_t)g * a.vs[1] + (int64_t)slot0 * a.vs[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                kf[mb][ks] = *(const bf16x8*)(kb + (int64_t)(tau0 + 4 * mb) * a.ks[2] + 32 * ks + 8 * lq);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = i * 64 + lane;
            const int tk = c >> 4;
            const int d8 = (c & 15) * 8;
            vr[i] = (tok0 + tk < end) ? *(const uint4*)(vb + (int64_t)tk * a.vs[2] + d8)
                                      : uint4{0u, 0u, 0u, 0u};
        }
    };

    if (b0 < b1) load_step(b0);
    for (int blk = b0; blk < b1; ++blk) {
        const int tok0 = start + blk * kStep;
        // stage V (keys past the split end are zero) and keep K in registers
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = i * 64 + lane;
            const int tk = c >> 4;
            const int d8 = (c & 15) * 8;
            uint2* dst = (uint2*)(vt + tk * kVPitch + d8 * 2);
            dst[0] = uint2{vr[i].x, vr[i].y};
            dst[1] = uint2{vr[i].z, vr[i].w};
        }
        bf16x8 kcur[2][4];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) kcur[mb][ks] = kf[mb][ks];
        if (blk + 1 < b1) load_step(blk + 1);
        wave_lds_sync();

        bf16x8 pf[kNT];
#pragma unroll
        for (int i = 0; i < kNT; ++i) {
            if (i < nt) {
                f32x4 sc[2];
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    f32x4 c4 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks)
                        c4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kcur[mb][ks], qf[i][ks], c4, 0, 0, 0);
                    sc[mb] = c4;
                }
                float sv[8];
                float bm = -__builtin_huge_valf();
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int key = tok0 + 8 * lq + 4 * mb + e;
                        const bool ok = key < end && key <= lim[i];
                        const float v = ok ? sc[mb][e] * p.scale2 : -__builtin_huge_valf();
                        sv[4 * mb + e] = v;
                        bm = fmaxf(bm, v);
                    }
                bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
                bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
                const float mn = fmaxf(mrow[i], bm);
                float alpha = 1.0f;
                float pr[8];
                if (mn == -__builtin_huge_valf()) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) pr[k] = 0.0f;
                } else {
                    alpha = exp2f(mrow[i] - mn);
#pragma unroll
                    for (int k = 0; k < 8; ++k) pr[k] = exp2f(sv[k] - mn);
                }
                float ps = 0.0f;
#pragma unroll
                for (int k = 0; k < 8; ++k) ps += pr[k];
                lsum[i] = lsum[i] * alpha + ps;
                mrow[i] = mn;
#pragma unroll
                for (int db = 0; db < 8; ++db) acc[i][db] *= alpha;
                uint4 pk;
                pk.x = pack2_bf16(pr[0], pr[1]);
                pk.y = pack2_bf16(pr[2], pr[3]);
                pk.z = pack2_bf16(pr[4], pr[5]);
                pk.w = pack2_bf16(pr[6], pr[7]);
                pf[i] = __builtin_bit_cast(bf16x8, pk);
            }
        }
        // O^T[d, row] += V^T P^T: A = V[key 8*lq + i][d = 16*db + lr], read from LDS
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const unsigned char* col = vt + (16 * db + lr) * 2 + 8 * lq * kVPitch;
            uint16_t hv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) hv[i] = *(const uint16_t*)(col + i * kVPitch);
            uint4 pk;
            pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
            pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
            pk.z = (uint32_t)hv[4] | ((uint32_t)hv[5] << 16);
            pk.w = (uint32_t)hv[6] | ((uint32_t)hv[7] << 16);
            const bf16x8 vf = __builtin_bit_cast(bf16x8, pk);
#pragma unroll
            for (int i = 0; i < kNT; ++i)
                if (i < nt) acc[i][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[i], acc[i][db], 0, 0, 0);
        }
        wave_lds_sync();
    }

    // ---- combine the four waves (fixed order) -------------------------------
#pragma unroll
    for (int i = 0; i < kNT; ++i) {
        lsum[i] += __shfl_xor(lsum[i], 16, 64);
        lsum[i] += __shfl_xor(lsum[i], 32, 64);
        if (lq == 0) {
            s_m[wave][16 * i + lr] = mrow[i];
            s_l[wave][16 * i + lr] = lsum[i];
        }
    }
    __syncthreads();
    float Mrow[kNT], Lrow[kNT];
#pragma unroll
    for (int i = 0; i < kNT; ++i) {
        const int rr = 16 * i + lr;
        float M = s_m[0][rr];
#pragma unroll
        for (int w = 1; w < kMfWaves; ++w) M = fmaxf(M, s_m[w][rr]);
        float L = 0.0f;
#pragma unroll
        for (int w = 0; w < kMfWaves; ++w)
            if (s_m[w][rr] > -__builtin_huge_valf()) L += s_l[w][rr] * exp2f(s_m[w][rr] - M);
        const float f = mrow[i] > -__builtin_huge_valf() ? exp2f(mrow[i] - M) : 0.0f;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[i][db] *= f;
        Mrow[i] = M;
        Lrow[i] = L;
    }
    float* ob = (float*)lds;  // [d][kOPitch]
    for (int w = kMfWaves - 1; w >= 0; --w) {
        if (wave == w) {
#pragma unroll
            for (int i = 0; i < kNT; ++i) {
                if (i < nt) {
#pragma unroll
                    for (int db = 0; db < 8; ++db)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            float* cell = ob + (16 * db + 4 * lq + e) * kOPitch + 16 * i + lr;
                            if (w == kMfWaves - 1) *cell = acc[i][db][e];
                            else if (w > 0) *cell = *cell + acc[i][db][e];
                            else acc[i][db][e] = acc[i][db][e] + *cell;
                        }
                }
            }
        }
        __syncthreads();
    }

    // ---- wave 0 writes the item's result -------------------------------------------
    uint16_t* outp = (uint16_t*)a.out;
    if (nsplit == 1) {
        if (wave == 0) {
#pragma unroll
            for (int i = 0; i < kNT; ++i) {
                const int row = row0 + 16 * i + lr;
                if (i < nt && row < rows) {
                    const int t = row / p.group;
                    const int h = g * p.group + (row - t * p.group);
                    const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
                    const float inv = 1.0f / Lrow[i];
#pragma unroll
                    for (int db = 0; db < 8; ++db) {
                        uint2 pk;
                        pk.x = pack2_bf16(acc[i][db][0] * inv, acc[i][db][1] * inv);
                        pk.y = pack2_bf16(acc[i][db][2] * inv, acc[i][db][3] * inv);
                        *(uint2*)(outp + orow * kD + 16 * db + 4 * lq) = pk;
                    }
                    if (a.lse && lq == 0) a.lse[orow] = (Mrow[i] + log2f(Lrow[i])) * kLn2;
                }
            }
        }
        return;
    }

    // ---- several splits: publish this split's partial, the last one merges ---------
    const int64_t slot_base = ((int64_t)rg * p.rc_max + rc) * p.max_splits;
    if (wave == 0) {
        float* part = p.part + (slot_base + s) * kSlotFloats;
#pragma unroll
        for (int i = 0; i < kNT; ++i) {
            const int rr = 16 * i + lr;
            if (i < nt) {
                if (lq == 0) {
                    part[rr] = Mrow[i];
                    part[kRows + rr] = Lrow[i];
                }
#pragma unroll
                for (int db = 0; db < 8; ++db)
                    *(f32x4*)(part + 2 * kRows + rr * kD + 16 * db + 4 * lq) = acc[i][db];
            }
        }
        __threadfence();
    }
    __syncthreads();
    if (tid == 0) {
        const int prev = atomicAdd(p.counters + (int64_t)rg * p.rc_max + rc, 1);
        s_last = prev == nsplit - 1;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    // merge: thread -> (row, quarter of d)
    const int mrow_i = tid >> 2;
    const int dq = (tid & 3) * 32;
    if (mrow_i < nrows) {
        const float* base = p.part + slot_base * kSlotFloats;
        float M = -__builtin_huge_valf();
        for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, base[sp * kSlotFloats + mrow_i]);
        float L = 0.0f;
        float o[32];
#pragma unroll
        for (int k = 0; k < 32; ++k) o[k] = 0.0f;
        for (int sp = 0; sp < nsplit; ++sp) {
            const float* sl = base + sp * kSlotFloats;
            const float ms = sl[mrow_i];
            if (!(ms > -__builtin_huge_valf())) continue;
            const float f = exp2f(ms - M);
            L += sl[kRows + mrow_i] * f;
            const f32x4* src = (const f32x4*)(sl + 2 * kRows + mrow_i * kD + dq);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const f32x4 v = src[k];
                o[4 * k + 0] += v[0] * f;
                o[4 * k + 1] += v[1] * f;
                o[4 * k + 2] += v[2] * f;
                o[4 * k + 3] += v[3] * f;
            }
        }
        const int row = row0 + mrow_i;
        const int t = row / p.group;
        const int h = g * p.group + (row - t * p.group);
        const int64_t orow = (int64_t)(q0 + t) * a.Hq + h;
        const float inv = 1.0f / L;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            uint2 pk;
            pk.x = pack2_bf16(o[4 * k] * inv, o[4 * k + 1] * inv);
            pk.y = pack2_bf16(o[4 * k + 2] * inv, o[4 * k + 3] * inv);
            *(uint2*)(outp + orow * kD + dq + 4 * k) = pk;
        }
        if (a.lse && dq == 0) a.lse[orow] = (M + log2f(L)) * kLn2;
    }
}

hipError_t launch_attn_mfma(const AttnArgs& a, void* ws, hipStream_t s) {
    const MfGeom g = mf_geom(a);
    MfParams p;
    p.a = a;
    p.group = g.group;
    p.max_splits = g.max_splits;
    p.rc_max = g.rc_max;
    p.n_items = g.n_items;
    p.scale2 = a.scale * kLog2e;
    p.counters = (int*)ws;
    p.part = (float*)((char*)ws + g.counter_bytes);
    const int n_counters = a.R * a.Hkv * g.rc_max;
    hipLaunchKernelGGL(mf_zero, dim3(std::min(1024, (n_counters + 255) / 256)), dim3(256), 0, s,
                       p.counters, n_counters);
    const int64_t grid = ((g.n_items + 7) / 8) * 8 * g.rc_max;
    hipLaunchKernelGGL(attn_mfma_kernel, dim3((unsigned)grid), dim3(kMfThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace dspark

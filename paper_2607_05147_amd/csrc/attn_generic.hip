// Ragged causal verify attention over a paged KV cache, vector-ALU path.
//
// Handles fp32 and bf16 and any head size that is a multiple of 8 (up to 576),
// including latent attention where the values alias the keys.  One wave per
// work item (query token, KV head, block of up to 8 query heads of that KV
// head's group, KV split): each lane owns one key of a 64-key tile for the
// score/softmax step and a slice of the value dimension for the weighted sum.
// Every split writes (max, sum, unnormalised output) for its rows; a merge
// kernel combines the splits in order, so results are bitwise reproducible.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"

namespace dspark {

constexpr int kGenHB = 8;          // query heads per work item
constexpr int kGenMaxD = 576;      // largest head dim
constexpr int kGenDPL = kGenMaxD / DSPARK_WAVE;  // value dims per lane (9)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

static int gen_splits(const AttnArgs& a) {
    const int64_t max_kv = (int64_t)a.max_pages * a.page;
    const int64_t s = (max_kv + 1023) / 1024;
    return (int)std::min<int64_t>(std::max<int64_t>(s, 1), 8);
}

size_t attn_generic_workspace(const AttnArgs& a) {
    const size_t rows = (size_t)a.R * a.max_q * a.Hq;
    return rows * gen_splits(a) * (size_t)(a.Dv + 2) * sizeof(float);
}

struct GenParams {
    AttnArgs a;
    int splits;
    int nhb;      // head blocks per KV head
    int group;
    float scale2; // scale * log2(e)
    float* part;  // [R*max_q][Hq][splits][Dv + 2]
};

// flattened verify tokens, clamped to the R * max_q rows the caller sized for
__device__ __forceinline__ int cu_q_total(const AttnArgs& a) {
    const int t = a.cu_q[a.R];
    const int mx = a.R * a.max_q;
    return t < 0 ? 0 : (t > mx ? mx : t);
}

// Request r's first row q0, row count ql and context kv; false when the
// request is malformed: ql outside [1, max_q], kv outside [ql, max_pages *
// page], or rows outside [0, min(cu_q[R], R * max_q)).  The grid is indexed by
// slot = r * max_q + t, so no token -> request search depends on cu_q being
// ordered.
__device__ __forceinline__ bool gen_request(const AttnArgs& a, int r, int& q0, int& ql, int& kv) {
    q0 = a.cu_q[r];
    ql = a.cu_q[r + 1] - q0;
    kv = a.kv_len[r];
    if (ql < 1 || ql > a.max_q || kv < ql || kv > a.max_pages * a.page) return false;
    return q0 >= 0 && (int64_t)q0 + ql <= cu_q_total(a);
}

template <typename T>
__global__ __launch_bounds__(DSPARK_WAVE) void attn_generic_kernel(GenParams p) {
    const AttnArgs& a = p.a;
    __shared__ float qs[kGenHB][kGenMaxD];
    const int lane = threadIdx.x;
    int64_t b = blockIdx.x;
    const int s = (int)(b % p.splits); b /= p.splits;
    const int hb = (int)(b % p.nhb);   b /= p.nhb;
    const int g = (int)(b % a.Hkv);    b /= a.Hkv;
    const int slot = (int)b;  // r * max_q + t
    const int r = slot / a.max_q;
    const int t = slot - r * a.max_q;
    int q0, ql, kv;
    if (!gen_request(a, r, q0, ql, kv) || t >= ql) return;
    const int tok = q0 + t;
    const int visible = kv - ql + t + 1;
    const int h0 = g * p.group + hb * kGenHB;
    const int nh = min(kGenHB, p.group - hb * kGenHB);
    // this split's key range
    const int per = ((visible + p.splits - 1) / p.splits + 15) & ~15;
    const int k_begin = min(visible, s * per);
    const int k_end = min(visible, k_begin + per);

    const T* q = (const T*)a.q;
    const T* kc = (const T*)a.k;
    const T* vc = (const T*)a.v;
    for (int i = lane; i < kGenHB * a.Dqk; i += DSPARK_WAVE) {
        const int hh = i / a.Dqk, d = i % a.Dqk;
        qs[hh][d] = hh < nh ? Elem<T>::load(q, ((int64_t)tok * a.Hq + h0 + hh) * a.Dqk + d) *
                                  p.scale2
                            : 0.0f;
    }
    __syncthreads();

    float m[kGenHB], l[kGenHB], o[kGenHB][kGenDPL];
#pragma unroll
    for (int hh = 0; hh < kGenHB; ++hh) {
        m[hh] = -__builtin_huge_valf();
        l[hh] = 0.0f;
#pragma unroll
        for (int e = 0; e < kGenDPL; ++e) o[hh][e] = 0.0f;
    }
    const int32_t* bt = a.block_table + (int64_t)r * a.max_pages;
    for (int k0 = k_begin; k0 < k_end; k0 += DSPARK_WAVE) {
        const int j = k0 + lane;
        const bool valid = j < k_end;
        float sc[kGenHB];
#pragma unroll
        for (int hh = 0; hh < kGenHB; ++hh) sc[hh] = 0.0f;
        if (valid) {
            const int64_t page = bt[j / a.page];
            const T* kr = kc + page * a.ks[0] + g * a.ks[1] + (int64_t)(j % a.page) * a.ks[2];
            for (int d = 0; d < a.Dqk; ++d) {
                const float kd = Elem<T>::load(kr, d);
#pragma unroll
                for (int hh = 0; hh < kGenHB; ++hh) sc[hh] += qs[hh][d] * kd;
            }
        }
        float pr[kGenHB];
#pragma unroll
        for (int hh = 0; hh < kGenHB; ++hh) {
            const float sv = valid ? sc[hh] : -__builtin_huge_valf();
            const float mt = wave_max(sv);
            const float mn = fmaxf(m[hh], mt);
            const float alpha = m[hh] == -__builtin_huge_valf() ? 0.0f : exp2f(m[hh] - mn);
            pr[hh] = valid ? exp2f(sv - mn) : 0.0f;
            l[hh] = l[hh] * alpha + wave_sum(pr[hh]);
            m[hh] = mn;
#pragma unroll
            for (int e = 0; e < kGenDPL; ++e) o[hh][e] *= alpha;
        }
        const int nvalid = min(DSPARK_WAVE, k_end - k0);
        for (int jj = 0; jj < nvalid; ++jj) {
            const int key = k0 + jj;
            const int64_t page = bt[key / a.page];
            const T* vr = vc + page * a.vs[0] + g * a.vs[1] + (int64_t)(key % a.page) * a.vs[2];
            float pj[kGenHB];
#pragma unroll
            for (int hh = 0; hh < kGenHB; ++hh) pj[hh] = __shfl(pr[hh], jj, DSPARK_WAVE);
#pragma unroll
            for (int e = 0; e < kGenDPL; ++e) {
                const int d = lane + e * DSPARK_WAVE;
                if (d < a.Dv) {
                    const float vd = Elem<T>::load(vr, d);
#pragma unroll
                    for (int hh = 0; hh < kGenHB; ++hh) o[hh][e] += pj[hh] * vd;
                }
            }
        }
    }
    // partial for (slot, h, s): [m, l, o[0..Dv)]
    for (int hh = 0; hh < nh; ++hh) {
        float* dst = p.part + (((int64_t)slot * a.Hq + h0 + hh) * p.splits + s) * (a.Dv + 2);
        if (lane == 0) { dst[0] = m[hh]; dst[1] = l[hh]; }
#pragma unroll
        for (int e = 0; e < kGenDPL; ++e) {
            const int d = lane + e * DSPARK_WAVE;
            if (d < a.Dv) dst[2 + d] = o[hh][e];
        }
    }
}

template <typename T>
__global__ __launch_bounds__(256) void attn_generic_merge(GenParams p) {
    const AttnArgs& a = p.a;
    const int64_t prow = (int64_t)blockIdx.x;  // (slot, h)
    const int slot = (int)(prow / a.Hq);
    const int h = (int)(prow - (int64_t)slot * a.Hq);
    const int r = slot / a.max_q;
    const int t = slot - r * a.max_q;
    int q0, ql, kv;
    if (!gen_request(a, r, q0, ql, kv) || t >= ql) return;
    const int64_t row = (int64_t)(q0 + t) * a.Hq + h;  // output row (token, head)
    const float* src = p.part + prow * p.splits * (a.Dv + 2);
    float M = -__builtin_huge_valf();
    for (int s = 0; s < p.splits; ++s) M = fmaxf(M, src[s * (a.Dv + 2)]);
    float L = 0.0f;
    for (int s = 0; s < p.splits; ++s) {
        const float ms = src[s * (a.Dv + 2)];
        if (ms > -__builtin_huge_valf()) L += src[s * (a.Dv + 2) + 1] * exp2f(ms - M);
    }
    const float invL = 1.0f / L;
    T* out = (T*)a.out;
    for (int d = threadIdx.x; d < a.Dv; d += blockDim.x) {
        float acc = 0.0f;
        for (int s = 0; s < p.splits; ++s) {
            const float ms = src[s * (a.Dv + 2)];
            if (ms > -__builtin_huge_valf()) acc += src[s * (a.Dv + 2) + 2 + d] * exp2f(ms - M);
        }
        Elem<T>::store(out, row * a.Dv + d, acc * invL);
    }
    if (a.lse && threadIdx.x == 0) a.lse[row] = (M + log2f(L)) * kLn2;
}

hipError_t launch_attn_generic(const AttnArgs& a, void* ws, hipStream_t s) {
    GenParams p;
    p.a = a;
    p.splits = gen_splits(a);
    p.group = a.Hq / a.Hkv;
    p.nhb = (p.group + kGenHB - 1) / kGenHB;
    p.scale2 = a.scale * kLog2e;
    p.part = (float*)ws;
    const int64_t tokens = (int64_t)a.R * a.max_q;
    const int64_t items = tokens * a.Hkv * p.nhb * p.splits;
    if (a.bf16)
        hipLaunchKernelGGL(attn_generic_kernel<uint16_t>, dim3((unsigned)items), dim3(DSPARK_WAVE),
                           0, s, p);
    else
        hipLaunchKernelGGL(attn_generic_kernel<float>, dim3((unsigned)items), dim3(DSPARK_WAVE), 0,
                           s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t rows = tokens * a.Hq;
    if (a.bf16)
        hipLaunchKernelGGL(attn_generic_merge<uint16_t>, dim3((unsigned)rows), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(attn_generic_merge<float>, dim3((unsigned)rows), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace dspark

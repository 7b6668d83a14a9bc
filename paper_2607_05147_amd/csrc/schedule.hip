// Hardware-aware prefix scheduler (Algorithm 1 of the section on
// confidence-scheduled verification) as one gfx950 workgroup.
//
// Steps, all on the device so the verification step needs no host round trip:
//   1. survival a[r][j] = prod_{i<=j} c[r][i] (fp64, multiplied in increasing j;
//      the same sequence of roundings on every implementation);
//   2. bitonic sort of the R*K candidates in LDS, descending a, ties by (r, j):
//      the key is the bit pattern of a (non-negative doubles order like their
//      bits) plus the flat index r*K + j;
//   3. block-wide fp64 inclusive scan of the sorted a: tau_n = R + sum_{m<=n} a_m;
//   4. Theta_n = tau_n * SPS(R + n + 1); mode 0 stops at the first n whose Theta
//      does not exceed its predecessor's (Theta_{-1} = R * SPS(R)), mode 1 takes
//      the first maximum;
//   5. len[r] = the largest admitted position of r (admission follows each
//      request's prefix order, since a is non-increasing in j), then cu_q and the
//      token -> request marker.
#include "device_common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace dspark {

constexpr int kSchedThreads = 1024;
constexpr int kSchedWaves = kSchedThreads / DSPARK_WAVE;

static int next_pow2(int n) {
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

size_t schedule_lds_bytes(int R, int K) {
    const int N = R * K;
    const int Np = next_pow2(N > 0 ? N : 1);
    size_t b = (size_t)Np * 8 + (size_t)Np * 2;
    b = (b + 15) & ~(size_t)15;
    b += (size_t)R * 4;
    b = (b + 15) & ~(size_t)15;
    b += (size_t)(N > 0 ? N : 1) * 4;  // staged confidences
    return b;
}

__device__ __forceinline__ double sched_conf(float c) {
    if (!(c > 0.0f)) return 0.0;
    if (c > 1.0f) return 1.0;
    return (double)c;
}

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(
    const float* __restrict__ conf, int R, int K, const double* __restrict__ sps, int mode,
    int Np, int32_t* __restrict__ len_out, int32_t* __restrict__ cu_q,
    int32_t* __restrict__ tok_req) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint64_t* key = reinterpret_cast<uint64_t*>(smem);
    uint16_t* idx = reinterpret_cast<uint16_t*>(key + Np);
    const size_t len_off = (((size_t)Np * 10) + 15) & ~(size_t)15;
    int32_t* lenl = reinterpret_cast<int32_t*>(smem + len_off);
    float* confl = reinterpret_cast<float*>(smem + ((len_off + (size_t)R * 4 + 15) & ~(size_t)15));

    __shared__ double s_wave_tot[kSchedWaves];
    __shared__ int s_first;
    __shared__ int s_ncand;
    __shared__ double s_best_v[kSchedWaves];
    __shared__ int s_best_n[kSchedWaves];
    __shared__ int s_wave_int[kSchedWaves];

    const int tid = threadIdx.x;
    const int lane = tid & (DSPARK_WAVE - 1);
    const int wave = tid / DSPARK_WAVE;
    const int N = R * K;

    if (tid == 0) s_ncand = 0;
    __syncthreads();

    // 1. survival products, one request per thread; the confidences are first
    // staged in LDS with coalesced loads
    for (int i = tid; i < N; i += kSchedThreads) confl[i] = conf[i];
    __syncthreads();
    int my_cand = 0;
    for (int r = tid; r < R; r += kSchedThreads) {
        double p = 1.0;
        for (int j = 0; j < K; ++j) {
            p = p * sched_conf(confl[r * K + j]);
            key[r * K + j] = (uint64_t)__double_as_longlong(p);
            idx[r * K + j] = (uint16_t)(r * K + j);
            my_cand += p > 0.0;
        }
        lenl[r] = 0;
    }
    for (int i = N + tid; i < Np; i += kSchedThreads) {
        key[i] = 0;
        idx[i] = 0xFFFF;
    }
    if (my_cand) atomicAdd(&s_ncand, my_cand);
    __syncthreads();

    // 2. bitonic sort: "x before y" iff key_x > key_y, or equal keys and idx_x < idx_y
    for (int k = 2; k <= Np; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < Np; i += kSchedThreads) {
                const int p = i ^ j;
                if (p > i) {
                    const uint64_t ki = key[i], kp = key[p];
                    const uint16_t ii = idx[i], ip = idx[p];
                    const bool p_first = (kp > ki) || (kp == ki && ip < ii);
                    const bool up = (i & k) == 0;
                    if (up ? p_first : !p_first) {
                        key[i] = kp; key[p] = ki;
                        idx[i] = ip; idx[p] = ii;
                    }
                }
            }
            __syncthreads();
        }
    }
    const int ncand = s_ncand;

    // 3. inclusive scan of the sorted survival probabilities (fp64)
    const int seg = Np >= kSchedThreads ? Np / kSchedThreads : 1;  // <= 8
    const int base = tid * seg;
    double loc[8];
    double run = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        if (e < seg) {
            const int n = base + e;
            const double a = (n < ncand) ? __longlong_as_double((long long)key[n]) : 0.0;
            run = run + a;
            loc[e] = run;
        }
    }
    // wave inclusive scan of the per-thread totals
    double incl = run;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const double t = __shfl_up(incl, o, DSPARK_WAVE);
        if (lane >= o) incl = incl + t;
    }
    if (lane == DSPARK_WAVE - 1) s_wave_tot[wave] = incl;
    __syncthreads();
    double wave_off = 0.0;
    for (int w = 0; w < wave; ++w) wave_off = wave_off + s_wave_tot[w];
    const double excl = wave_off + (incl - run);
    __syncthreads();  // every thread has read its elements' keys
    const double Rd = (double)R;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        if (e < seg) {
            const int n = base + e;
            if (n < ncand) key[n] = (uint64_t)__double_as_longlong(Rd + (excl + loc[e]));
        }
    }
    if (tid == 0) s_first = ncand;
    __syncthreads();

    // 4. throughput along the greedy path and the stop rule
    const double theta0 = Rd * sps[R];
    int n_adm;
    if (mode == 0) {
        int first = ncand;
        for (int e = 0; e < seg; ++e) {
            const int n = base + e;
            if (n >= ncand) break;
            const double th = __longlong_as_double((long long)key[n]) * sps[R + n + 1];
            const double prev = n == 0
                ? theta0
                : __longlong_as_double((long long)key[n - 1]) * sps[R + n];
            if (!(th > prev)) { first = n; break; }
        }
        if (first < ncand) atomicMin(&s_first, first);
        __syncthreads();
        n_adm = s_first;
    } else {
        double bv = tid == 0 ? theta0 : -1.0 / 0.0;
        int bn = -1;
        for (int e = 0; e < seg; ++e) {
            const int n = base + e;
            if (n >= ncand) break;
            const double th = __longlong_as_double((long long)key[n]) * sps[R + n + 1];
            if (th > bv) { bv = th; bn = n; }
        }
        if (tid != 0 && bn == -1) bn = 0x7fffffff;
#pragma unroll
        for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
            const double ov = __shfl_xor(bv, o, DSPARK_WAVE);
            const int on = __shfl_xor(bn, o, DSPARK_WAVE);
            if (ov > bv || (ov == bv && on < bn)) { bv = ov; bn = on; }
        }
        if (lane == 0) { s_best_v[wave] = bv; s_best_n[wave] = bn; }
        __syncthreads();
        if (tid == 0) {
            double v = s_best_v[0];
            int n = s_best_n[0];
            for (int w = 1; w < kSchedWaves; ++w)
                if (s_best_v[w] > v || (s_best_v[w] == v && s_best_n[w] < n)) {
                    v = s_best_v[w];
                    n = s_best_n[w];
                }
            s_first = n + 1;
        }
        __syncthreads();
        n_adm = s_first;
    }

    // 5. lengths: the largest admitted position of each request
    for (int n = tid; n < n_adm; n += kSchedThreads) {
        const int i = idx[n];
        atomicMax(&lenl[i / K], i % K + 1);
    }
    __syncthreads();

    // cu_q: exclusive scan of 1 + len over requests (contiguous ranges per thread)
    const int per = (R + kSchedThreads - 1) / kSchedThreads;
    const int r0 = tid * per;
    const int r1 = min(R, r0 + per);
    int tot = 0;
    for (int r = r0; r < r1; ++r) tot += 1 + lenl[r];
    int iinc = tot;
#pragma unroll
    for (int o = 1; o < DSPARK_WAVE; o <<= 1) {
        const int t = __shfl_up(iinc, o, DSPARK_WAVE);
        if (lane >= o) iinc += t;
    }
    if (lane == DSPARK_WAVE - 1) s_wave_int[wave] = iinc;
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave; ++w) off += s_wave_int[w];
    off += iinc - tot;
    for (int r = r0; r < r1; ++r) {
        const int q = 1 + lenl[r];
        len_out[r] = lenl[r];
        if (cu_q) cu_q[r] = off;
        if (tok_req)
            for (int t = 0; t < q; ++t) tok_req[off + t] = r;
        off += q;
    }
    if (r1 == R && r0 < r1) {
        if (cu_q) cu_q[R] = off;
    }
    if (R == 0 && tid == 0 && cu_q) cu_q[0] = 0;
    if (tok_req) {
        __syncthreads();
        // total = sum(1 + len) is known to the thread owning the last request;
        // recompute it from the scan totals so every thread can clear the tail
        int total = 0;
        for (int w = 0; w < kSchedWaves; ++w) total += s_wave_int[w];
        for (int i = total + tid; i < R * (K + 1); i += kSchedThreads) tok_req[i] = -1;
    }
}

hipError_t launch_schedule(const float* conf, int R, int K, const double* sps, int mode,
                           int32_t* len, int32_t* cu_q, int32_t* tok_req, hipStream_t s) {
    const int N = R * K;
    const int Np = next_pow2(N > 0 ? N : 1);
    const size_t lds = schedule_lds_bytes(R, K);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)schedule_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(kSchedThreads), lds, s, conf, R, K, sps,
                       mode, Np, len, cu_q, tok_req);
    return hipGetLastError();
}

}  // namespace dspark

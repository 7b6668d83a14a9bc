// Input checks for the device-side values of the three stages and the draft
// block.
//
// The stages clamp what lives in device memory (row offsets, context
// lengths, tokens) so that no access leaves the caller's buffers, and skip
// requests whose values break the documented rules.  Two things cannot be
// clamped: a block-table entry names a page of a cache whose size the call is
// not told, and a uniform, confidence or temperature outside its range
// silently changes the result.  These kernels look at the values before a call and report the
// first rule broken (smallest request, then the rule's order below) as four
// int32 {code, request, index, value bits}; code 0 means none.  One
// workgroup walks the requests 256 at a time; it reads only the arrays and
// sizes it is given.
#include "device_common.h"
#include "kernels.h"

namespace dspark {

namespace {
constexpr int kChkThreads = 256;

// The workgroup's first finding: every thread proposes (request, code,
// index, value) for its own request, the smallest request wins.
struct Finding {
    int code, r, i, v;
};

__device__ void report_first(const Finding& f, int32_t* report, bool& done) {
    __shared__ int s_first;
    if (threadIdx.x == 0) s_first = 0x7fffffff;
    __syncthreads();
    if (f.code) atomicMin(&s_first, f.r);
    __syncthreads();
    const int first = s_first;
    if (first != 0x7fffffff) {
        if (f.code && f.r == first) {
            report[0] = f.code;
            report[1] = f.r;
            report[2] = f.i;
            report[3] = f.v;
        }
        done = true;
    }
    __syncthreads();  // s_first is rewritten by the next round
}
}  // namespace

// Verify-attention inputs: 1 rows of request r outside [0, min(cu_q[R],
// R*max_q)) or cu_q decreasing (index 0: cu_q[r], 1: cu_q[r+1]); 2 q_len above
// max_q; 3 kv_len outside [q_len, max_pages*page_size]; 4 a block-table entry
// of a page the request reads outside [0, num_pages) (index: logical page).
__global__ __launch_bounds__(kChkThreads) void chk_verify(const int32_t* block_table, int max_pages,
                                                          const int32_t* kv_len, const int32_t* cu_q, int R,
                                                          int max_q, int page_size, int num_pages,
                                                          int32_t* report) {
    const int64_t total = min((int64_t)cu_q[R], (int64_t)R * max_q);
    bool done = false;
    for (int base = 0; base < R && !done; base += kChkThreads) {
        const int r = base + (int)threadIdx.x;
        Finding f{0, r, 0, 0};
        if (r < R) {
            const int q0 = cu_q[r], q1 = cu_q[r + 1];
            const int ql = q1 - q0;
            const int kv = kv_len[r];
            if (q0 < 0 || q1 < q0 || (int64_t)q1 > total) {
                f = Finding{1, r, q0 < 0 ? 0 : 1, q0 < 0 ? q0 : q1};
            } else if (ql > max_q) {
                f = Finding{2, r, 0, ql};
            } else if (kv < ql || (int64_t)kv > (int64_t)max_pages * page_size) {
                f = Finding{3, r, 0, kv};
            } else {
                const int np = (int)(((int64_t)kv + page_size - 1) / page_size);
                for (int p = 0; p < np; ++p) {
                    const int e = block_table[(int64_t)r * max_pages + p];
                    if (e < 0 || e >= num_pages) {
                        f = Finding{4, r, p, e};
                        break;
                    }
                }
            }
        }
        report_first(f, report, done);
    }
    if (!done && threadIdx.x == 0) report[0] = report[1] = report[2] = report[3] = 0;
}

// Acceptance inputs: 1 rows of request r outside [0, min(cu_q[R], R*(K+1)))
// or cu_q decreasing; 2 len_r = q_len - 1 outside [0, K]; 3 a uniform u[r, t]
// (t = 0 .. K) outside [0, 1) or NaN (index t, value: its bits).
__global__ __launch_bounds__(kChkThreads) void chk_accept(const int32_t* cu_q, const float* u, int R, int K,
                                                          int32_t* report) {
    const int64_t total = min((int64_t)cu_q[R], (int64_t)R * (K + 1));
    bool done = false;
    for (int base = 0; base < R && !done; base += kChkThreads) {
        const int r = base + (int)threadIdx.x;
        Finding f{0, r, 0, 0};
        if (r < R) {
            const int q0 = cu_q[r], q1 = cu_q[r + 1];
            const int len = q1 - q0 - 1;
            if (q0 < 0 || q1 < q0 || (int64_t)q1 > total) {
                f = Finding{1, r, q0 < 0 ? 0 : 1, q0 < 0 ? q0 : q1};
            } else if (len < 0 || len > K) {
                f = Finding{2, r, 0, len};
            } else if (u) {
                for (int t = 0; t <= K; ++t) {
                    const float x = u[(int64_t)r * (K + 1) + t];
                    if (!(x >= 0.0f && x < 1.0f)) {
                        f = Finding{3, r, t, (int)__float_as_uint(x)};
                        break;
                    }
                }
            }
        }
        report_first(f, report, done);
    }
    if (!done && threadIdx.x == 0) report[0] = report[1] = report[2] = report[3] = 0;
}

// Scheduler inputs: 1 a confidence conf[r, j] outside [0, 1] or NaN (index j,
// value: its bits).
__global__ __launch_bounds__(kChkThreads) void chk_schedule(const float* conf, int R, int K, int32_t* report) {
    bool done = false;
    for (int base = 0; base < R && !done; base += kChkThreads) {
        const int r = base + (int)threadIdx.x;
        Finding f{0, r, 0, 0};
        if (r < R) {
            for (int j = 0; j < K; ++j) {
                const float x = conf[(int64_t)r * K + j];
                if (!(x >= 0.0f && x <= 1.0f)) {
                    f = Finding{1, r, j, (int)__float_as_uint(x)};
                    break;
                }
            }
        }
        report_first(f, report, done);
    }
    if (!done && threadIdx.x == 0) report[0] = report[1] = report[2] = report[3] = 0;
}

// Drafter inputs: 1 a per-position temperature T_k outside (0, inf) or NaN
// (request -1, index k, value: its bits); 2 a uniform u[r, k] outside [0, 1)
// or NaN (index k, value: its bits).
__global__ __launch_bounds__(kChkThreads) void chk_draft(const float* u, const float* sts_temp, int R, int K,
                                                         int32_t* report) {
    __shared__ int s_temp;  // first bad temperature (K if none)
    if (threadIdx.x == 0) s_temp = K;
    __syncthreads();
    if (sts_temp && (int)threadIdx.x < K) {
        const float t = sts_temp[threadIdx.x];
        if (!(t > 0.0f && t < __builtin_huge_valf())) atomicMin(&s_temp, (int)threadIdx.x);
    }
    __syncthreads();
    if (s_temp < K) {
        if (threadIdx.x == 0) {
            report[0] = 1;
            report[1] = -1;
            report[2] = s_temp;
            report[3] = (int)__float_as_uint(sts_temp[s_temp]);
        }
        return;
    }
    bool done = false;
    for (int base = 0; base < R && !done; base += kChkThreads) {
        const int r = base + (int)threadIdx.x;
        Finding f{0, r, 0, 0};
        if (r < R) {
            for (int k = 0; k < K; ++k) {
                const float x = u[(int64_t)r * K + k];
                if (!(x >= 0.0f && x < 1.0f)) {
                    f = Finding{2, r, k, (int)__float_as_uint(x)};
                    break;
                }
            }
        }
        report_first(f, report, done);
    }
    if (!done && threadIdx.x == 0) report[0] = report[1] = report[2] = report[3] = 0;
}

hipError_t launch_check_draft(const float* u, const float* sts_temp, int R, int K, int32_t* report,
                              hipStream_t s) {
    hipLaunchKernelGGL(chk_draft, dim3(1), dim3(kChkThreads), 0, s, u, sts_temp, R, K, report);
    return hipGetLastError();
}

hipError_t launch_check_verify(const int32_t* block_table, int max_pages, const int32_t* kv_len,
                               const int32_t* cu_q, int R, int max_q, int page_size, int num_pages,
                               int32_t* report, hipStream_t s) {
    hipLaunchKernelGGL(chk_verify, dim3(1), dim3(kChkThreads), 0, s, block_table, max_pages, kv_len, cu_q, R,
                       max_q, page_size, num_pages, report);
    return hipGetLastError();
}

hipError_t launch_check_accept(const int32_t* cu_q, const float* u, int R, int K, int32_t* report,
                               hipStream_t s) {
    hipLaunchKernelGGL(chk_accept, dim3(1), dim3(kChkThreads), 0, s, cu_q, u, R, K, report);
    return hipGetLastError();
}

hipError_t launch_check_schedule(const float* conf, int R, int K, int32_t* report, hipStream_t s) {
    hipLaunchKernelGGL(chk_schedule, dim3(1), dim3(kChkThreads), 0, s, conf, R, K, report);
    return hipGetLastError();
}

}  // namespace dspark

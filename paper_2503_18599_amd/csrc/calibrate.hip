// Offline outlier-threshold profiling (Oaken Sec. 4.3, "offline outlier threshold
// profiling"; ratios of Sec. 6.1).
//
// The paper takes topK boundaries per profiling run and averages them.  Here every
// boundary is an exact order statistic of fp16 data, found without sorting: fp16 bit
// patterns map to 16-bit keys whose integer order is the value order (or the
// magnitude order), and a two-pass radix select over the high then the low key byte
// finds the key of a given rank with 256-bin LDS histograms.
#include "oaken_internal.h"

#include <hip/hip_fp16.h>

namespace oaken {
namespace {

constexpr int kCalThreads = 512;

// Monotone key for value order: negative patterns are reversed below positive ones.
__device__ inline uint32_t value_key(uint16_t b) {
    return (b & 0x8000u) ? (uint32_t)(~b & 0xffffu) : (uint32_t)(b | 0x8000u);
}
__device__ inline uint16_t value_key_inverse(uint32_t k) {
    return (k & 0x8000u) ? (uint16_t)(k & 0x7fffu) : (uint16_t)(~k & 0xffffu);
}
// Magnitude order: drop the sign bit.
__device__ inline uint32_t mag_key(uint16_t b) { return b & 0x7fffu; }

// Three selections per (run, head, K|V): rank k_o and n-1-k_o in value order, rank
// k_i-1 in magnitude order.
__global__ __launch_bounds__(kCalThreads) void calib_select_kernel(CalibArgs a) {
    const int r = blockIdx.x, h = blockIdx.y, which = blockIdx.z;
    const uint16_t* src = which ? a.v : a.k;
    const int T = a.T, d = a.d, H = a.H;

    __shared__ uint32_t hist[3][256];
    __shared__ uint32_t sel_hi[3], sel_rank[3], sel_key[3];

    const int64_t rank[3] = {a.k_o, a.n - 1 - a.k_o, a.k_i > 0 ? a.k_i - 1 : 0};

    for (int pass = 0; pass < 2; ++pass) {
        for (int i = threadIdx.x; i < 3 * 256; i += blockDim.x) (&hist[0][0])[i] = 0;
        __syncthreads();
        for (int64_t i = threadIdx.x; i < a.n; i += blockDim.x) {
            const int t = (int)(i / d), j = (int)(i % d);
            const uint16_t b = src[(((int64_t)r * T + t) * H + h) * d + j];
            const uint32_t kv = value_key(b), km = mag_key(b);
            if (pass == 0) {
                atomicAdd(&hist[0][kv >> 8], 1u);
                atomicAdd(&hist[2][km >> 8], 1u);
            } else {
                if ((kv >> 8) == sel_hi[0]) atomicAdd(&hist[0][kv & 0xff], 1u);
                if ((kv >> 8) == sel_hi[1]) atomicAdd(&hist[1][kv & 0xff], 1u);
                if ((km >> 8) == sel_hi[2]) atomicAdd(&hist[2][km & 0xff], 1u);
            }
        }
        __syncthreads();
        if (threadIdx.x < 3) {
            const int q = threadIdx.x;
            const uint32_t* hq = (pass == 0 && q == 1) ? hist[0] : hist[q];
            const uint64_t want = (pass == 0) ? (uint64_t)rank[q] : (uint64_t)sel_rank[q];
            uint64_t acc = 0;
            int bin = 255;
            for (int k = 0; k < 256; ++k) {
                if (acc + hq[k] > want) { bin = k; break; }
                acc += hq[k];
            }
            if (pass == 0) {
                sel_hi[q] = (uint32_t)bin;
                sel_rank[q] = (uint32_t)(want - acc);
            } else {
                sel_key[q] = (sel_hi[q] << 8) | (uint32_t)bin;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        float* o = a.per_run + (((int64_t)r * H + h) * 2 + which) * 3;
        o[0] = __half2float(__ushort_as_half(value_key_inverse(sel_key[0])));
        o[1] = __half2float(__ushort_as_half(value_key_inverse(sel_key[1])));
        o[2] = (a.k_i > 0) ? __half2float(__ushort_as_half((uint16_t)sel_key[2])) : 0.0f;
    }
}

// fp64 mean over runs in run order, one fp32 rounding, ordering repair, -0 -> +0.
__global__ void calib_average_kernel(CalibArgs a) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;   // (head, which)
    if (i >= a.H * 2) return;
    double s_lo = 0.0, s_hi = 0.0, s_t = 0.0;
    for (int r = 0; r < a.R; ++r) {
        const float* o = a.per_run + ((int64_t)r * a.H * 2 + i) * 3;
        s_lo += (double)o[0];
        s_hi += (double)o[1];
        s_t += (double)o[2];
    }
    const float lo_o = (float)(s_lo / (double)a.R);
    const float hi_o = (float)(s_hi / (double)a.R);
    const float t = (float)(s_t / (double)a.R);
    float lo_i = fminf(fmaxf(-t, lo_o), hi_o);
    float hi_i = fmaxf(fminf(t, hi_o), lo_i);
    float v[4] = {lo_o, lo_i, hi_i, hi_o};
    for (int k = 0; k < 4; ++k) a.thr_out[i * 4 + k] = (v[k] == 0.0f) ? 0.0f : v[k];
}

}  // namespace

hipError_t launch_calibrate(const CalibArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(calib_select_kernel, dim3(a.R, a.H, 2), dim3(kCalThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(calib_average_kernel, dim3((a.H * 2 + 63) / 64), dim3(64), 0, st, a);
    return hipGetLastError();
}

}  // namespace oaken

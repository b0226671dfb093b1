// tas_pctl.hip - nearest-rank percentiles of the per-request latencies.
//
// For every instance and metric (TTFT, TTLT, max inter-token gap) the value
// at sorted position ceil(q*n/100) - 1 for q in {50, 90, 99}: the empirical
// t_p = inf{t : Fbar(t) <= (100-p)/100} (arXiv 2606.18431, Phase 4).
//
// One 256-thread workgroup per (instance, metric) runs an exact radix select
// over the 32-bit values, 11, 11 and 10 bits per pass, most significant digit
// first; the three ranks share each pass over the data (one LDS histogram of
// 2048 bins per rank; the first pass, where no prefix is fixed yet, needs
// only one). Integer work bound by HBM reads: 3 passes x 4 bytes per value,
// read 16 bytes per lane.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tas_internal.h"

namespace tas {
namespace {

constexpr int kThreads = 256;
constexpr int kPasses = 3;
constexpr int kBins = 2048;                 // 11-bit digits (the last pass: 10 bits)
constexpr int kShift[kPasses] = {21, 10, 0};
constexpr int kBits[kPasses] = {11, 11, 10};

__global__ __launch_bounds__(kThreads) void pctl_kernel(const uint32_t *ttft, const uint32_t *ttlt,
                                                        const uint32_t *tbt, int n_inst, int n,
                                                        uint32_t *out) {
    __shared__ uint32_t hist[3][kBins];
    __shared__ uint32_t pre[3];
    __shared__ int rk[3];
    const int b = blockIdx.x;
    const int inst = b / 3, metric = b % 3;
    if (inst >= n_inst) return;
    const uint32_t *v =
        (metric == 0 ? ttft : metric == 1 ? ttlt : tbt) + (size_t)inst * (size_t)n;
    const int tid = threadIdx.x;
    if (tid < 3) {
        const int q = tid == 0 ? 50 : tid == 1 ? 90 : 99;
        rk[tid] = (int)(((int64_t)q * n + 99) / 100);
        pre[tid] = 0;
    }
    for (int pass = 0; pass < kPasses; pass++) {
        const int sh = kShift[pass];
        const uint32_t dmask = (1u << kBits[pass]) - 1u;
        const int hs = sh + kBits[pass];  // bits above this digit: the fixed prefix
        for (int j = tid; j < 3 * kBins; j += kThreads) (&hist[0][0])[j] = 0;
        __syncthreads();
        const uint32_t p0 = pre[0], p1 = pre[1], p2 = pre[2];
        const auto count = [&](uint32_t x) {
            const uint32_t d = (x >> sh) & dmask;
            if (pass == 0) {
                atomicAdd(&hist[0][d], 1u);
            } else {
                const uint32_t hx = x >> hs;
                if (hx == (p0 >> hs)) atomicAdd(&hist[0][d], 1u);
                if (hx == (p1 >> hs)) atomicAdd(&hist[1][d], 1u);
                if (hx == (p2 >> hs)) atomicAdd(&hist[2][d], 1u);
            }
        };
        // 16-byte loads over the aligned body of the row, single values
        // before and after it
        const int head = (int)(((16u - ((uint32_t)(uintptr_t)v & 15u)) & 15u) >> 2);
        const int nh = head < n ? head : n;
        const int nv = (n - nh) >> 2;
        if (tid < nh) count(v[tid]);
        const uint4 *v4 = (const uint4 *)(v + nh);
        for (int i = tid; i < nv; i += kThreads) {
            const uint4 x = v4[i];
            count(x.x), count(x.y), count(x.z), count(x.w);
        }
        for (int i = nh + 4 * nv + tid; i < n; i += kThreads) count(v[i]);
        __syncthreads();
        // wave r < 3 finds rank r: each lane sums 32 consecutive bins, a wave
        // scan finds the lane whose bins hold the rank, that lane walks them
        const int wv = tid >> 6, ln = tid & 63;
        if (wv < 3) {
            const uint32_t *h = pass == 0 ? hist[0] : hist[wv];
            constexpr int kPer = kBins / 64;
            int s = 0;
            for (int j = 0; j < kPer; j++) s += (int)h[kPer * ln + j];
            int inc = s;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(inc, o);
                if (ln >= o) inc += y;
            }
            const int exc = inc - s;
            const int r = rk[wv];
            const uint64_t m = __ballot(exc < r && r <= inc);
            if (m) {
                const int src = __ffsll((unsigned long long)m) - 1;
                if (ln == src) {
                    int rr = r - exc, bin = kPer * ln;
                    for (int j = 0; j < kPer - 1; j++, bin++) {
                        const int c = (int)h[bin];
                        if (rr <= c) break;
                        rr -= c;
                    }
                    pre[wv] |= (uint32_t)bin << sh;
                    rk[wv] = rr;
                }
            }
        }
        __syncthreads();
    }
    if (tid < 3) out[(size_t)inst * 9 + metric * 3 + tid] = pre[tid];
}

}  // namespace
}  // namespace tas

int tas_launch_pctl(const uint32_t *ttft, const uint32_t *ttlt, const uint32_t *tbtmax,
                    int32_t n_inst, int32_t n_req, uint32_t *out, void *stream) {
    if (n_inst <= 0) return 0;
    hipLaunchKernelGGL(tas::pctl_kernel, dim3((unsigned)(3 * n_inst)), dim3(tas::kThreads), 0,
                       (hipStream_t)stream, ttft, ttlt, tbtmax, n_inst, n_req, out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

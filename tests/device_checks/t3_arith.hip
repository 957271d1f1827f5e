// Test-side device check: the Student-t draw's square root and division
// (cdt::t3_sqrt, cdt::t3_div from the library's own header) against the
// compiler's correctly rounded sqrtf and fp32 '/', bit for bit, on the
// ranges the draw reaches and beyond: every float in [2^-96, 2^7) for the
// square root, every divisor in [2^-17, 2^4) against 256 Irwin-Hall
// dividends (0 and +-n * 0x1.bb67aep-16 spread over n < 2^17) for the
// division.  The uncorrected forms (v_sqrt_f32 alone, a * v_rcp_f32(b)) are
// counted as well, to show the comparison can fail.  Prints one line per
// figure; exit status 0 when the program ran (the caller judges the counts).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "cdt_sim.hpp"

#pragma clang fp contract(off)

namespace {

constexpr uint32_t kSqrtLo = 0x0f800000u;  // 2^-96
constexpr uint32_t kSqrtHi = 0x43000000u;  // 2^7
constexpr uint32_t kDivLo = 0x37000000u;   // 2^-17
constexpr uint32_t kDivHi = 0x41800000u;   // 2^4
constexpr uint32_t kDividends = 256;

__global__ void sqrt_diff(uint32_t lo, uint32_t n, unsigned long long* out) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float x = __uint_as_float(lo + i);
    const uint32_t want = __float_as_uint(sqrtf(x));
    if (__float_as_uint(cdt::t3_sqrt(x)) != want) atomicAdd(&out[0], 1ull);
    if (__float_as_uint(__builtin_amdgcn_sqrtf(x)) != want) atomicAdd(&out[1], 1ull);
}

__global__ void div_diff(uint32_t lo, uint32_t n, const float* __restrict__ as,
                         unsigned long long* out) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float b = __uint_as_float(lo + i);
    uint32_t bad = 0, raw = 0;
    for (uint32_t k = 0; k < kDividends; ++k) {
        const float a = as[k];
        const uint32_t want = __float_as_uint(a / b);
        bad += __float_as_uint(cdt::t3_div(a, b)) != want;
        raw += __float_as_uint(a * __builtin_amdgcn_rcpf(b)) != want;
    }
    if (bad) atomicAdd(&out[0], static_cast<unsigned long long>(bad));
    if (raw) atomicAdd(&out[1], static_cast<unsigned long long>(raw));
}

#define CHECK(x)                                                                        \
    do {                                                                                \
        const hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                         \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            return 2;                                                                   \
        }                                                                               \
    } while (0)

}  // namespace

int main() {
    unsigned long long* cnt = nullptr;
    float* as = nullptr;
    CHECK(hipMalloc(&cnt, 2 * sizeof(unsigned long long)));
    CHECK(hipMalloc(&as, kDividends * sizeof(float)));
    float ha[kDividends];
    for (uint32_t k = 0; k < kDividends; ++k) {
        const int n = k == 0 ? 0 : static_cast<int>((k * 2654435761u) % 131071u);
        ha[k] = static_cast<float>((k & 1) ? n : -n) * 0x1.bb67aep-16f;
    }
    CHECK(hipMemcpy(as, ha, sizeof(ha), hipMemcpyHostToDevice));

    unsigned long long h[2] = {0, 0};
    CHECK(hipMemcpy(cnt, h, sizeof(h), hipMemcpyHostToDevice));
    const uint32_t ns = kSqrtHi - kSqrtLo;
    hipLaunchKernelGGL(sqrt_diff, dim3((ns + 255) / 256), dim3(256), 0, 0, kSqrtLo, ns, cnt);
    CHECK(hipGetLastError());
    CHECK(hipMemcpy(h, cnt, sizeof(h), hipMemcpyDeviceToHost));
    printf("sqrt_inputs %u\nsqrt_differ %llu\nsqrt_raw_differ %llu\n", ns, h[0], h[1]);
    fflush(stdout);

    h[0] = h[1] = 0;
    CHECK(hipMemcpy(cnt, h, sizeof(h), hipMemcpyHostToDevice));
    const uint32_t slice = 1u << 24;
    for (uint32_t s = kDivLo; s < kDivHi; s += slice) {
        const uint32_t n = kDivHi - s < slice ? kDivHi - s : slice;
        hipLaunchKernelGGL(div_diff, dim3((n + 255) / 256), dim3(256), 0, 0, s, n, as, cnt);
        CHECK(hipGetLastError());
    }
    CHECK(hipMemcpy(h, cnt, sizeof(h), hipMemcpyDeviceToHost));
    printf("div_pairs %llu\ndiv_differ %llu\ndiv_raw_differ %llu\n",
           static_cast<unsigned long long>(kDivHi - kDivLo) * kDividends, h[0], h[1]);
    CHECK(hipFree(cnt));
    CHECK(hipFree(as));
    return 0;
}

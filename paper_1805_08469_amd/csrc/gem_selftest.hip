// gem_selftest.hip -- device self-tests of the library's numerics (built as
// libgem_selftest.so; not part of the commit path).
//
// The commit kernels use range-specialised forms of correctly rounded
// division and square root (gem_device.hpp).  These kernels compare them, on
// the device and bit for bit, with hipcc's general IEEE operations:
//   - the logarithm's (f - 1) / (f + 1) (ln_quotient, and the general core
//     div_rn_core on the same operands) for every binary32 f the logarithm
//     can see (the 2^23 values in (sqrt(1/2), sqrt(2)]);
//   - the Box-Muller radius sqrt(-2 ln u) for every u = k 2^-24, k in
//     [1, 2^24];
//   - the guarded quotient div_rn on Philox-random operand pairs spread over
//     the whole binary32 range (zeros, subnormals, infinities and NaNs
//     included), and on every significand of the denominator against a set
//     of numerators.
// Each entry point returns GEM_OK and the number of mismatching results, or a
// GEM_E* code (bad argument, allocation or HIP failure).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gem.h"
#include "gem_device.hpp"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool same_bits(float x, float y)
{
    const bool both_nan = (x != x) && (y != y);
    return both_nan || __float_as_uint(x) == __float_as_uint(y);
}

// f in (sqrt(1/2), sqrt(2)]: index j < 2^23 takes 1.m with m = j (up to the
// sqrt(2) cut), j >= 2^23 takes 0.5 * 1.m; out-of-domain indices are skipped.
__global__ __launch_bounds__(kThreads) void ln_div_kernel(unsigned long long* bad)
{
    const uint32_t j = blockIdx.x * kThreads + threadIdx.x;   // grid covers 2^24 exactly
    const uint32_t mant = j & 0x007FFFFFu;
    const bool upper = j >= (1u << 23);
    if (upper != (mant > 0x003504F3u)) return;   // the logarithm picks the branch by mant
    const float f = __uint_as_float(mant | (upper ? 0x3F000000u : 0x3F800000u));
    const float a = f - 1.0f, b = f + 1.0f;
    const float want = a / b;
    // the two forms the library uses for this quotient
    if (!same_bits(gemk::ln_quotient(a, b), want)) atomicAdd(bad, 1ull);
    if (!same_bits(gemk::div_rn_core(a, b), want)) atomicAdd(bad, 1ull);
}

__global__ __launch_bounds__(kThreads) void radius_kernel(unsigned long long* bad)
{
    const uint32_t k = blockIdx.x * kThreads + threadIdx.x + 1u;   // 1 .. 2^24
    const float u = static_cast<float>(k) * 0x1p-24f;
    const float x = -2.0f * gemk::ln_of_unit(u);
    if (!same_bits(gemk::sqrt_rn_core(x), __builtin_sqrtf(x))) atomicAdd(bad, 1ull);
    // the two ways to the logarithm (from u, and from k with the scaling in
    // the exponent) agree
    if (!same_bits(gemk::ln_of_k24(k), gemk::ln_of_unit(u))) atomicAdd(bad, 1ull);
}

// A binary32 value from 32 random bits, with the exponent field drawn over
// its whole range (so every binade, subnormals, zeros, infinities and NaNs
// occur), or from a narrower window around 1.
__device__ __forceinline__ float spread(uint32_t x, uint32_t y, bool narrow)
{
    const uint32_t sign = x & 0x80000000u;
    const uint32_t mant = x & 0x007FFFFFu;
    uint32_t ex = narrow ? 127u - 70u + (y % 141u) : (y % 256u);
    return __uint_as_float(sign | (ex << 23) | mant);
}

__global__ __launch_bounds__(kThreads) void div_random_kernel(uint64_t seed, int64_t count,
                                                              unsigned long long* bad)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= count) return;
    const gemk::Words4 w = gemk::philox10(static_cast<uint32_t>(i), static_cast<uint32_t>(i >> 32),
                                          0x5e1f7e57u, 0u, static_cast<uint32_t>(seed),
                                          static_cast<uint32_t>(seed >> 32));
    const bool narrow = (w.x2 & 3u) != 0;   // three in four pairs near the core range
    const float num = spread(w.x0, w.x2 >> 2, narrow);
    const float den = spread(w.x1, w.x3, narrow);
    if (!same_bits(gemk::div_rn(num, den), num / den)) atomicAdd(bad, 1ull);
}

// Every significand of a denominator in [1, 2) scaled by 2^e_den, against
// numerators num[r].
__global__ __launch_bounds__(kThreads) void div_grid_kernel(const float* nums, int32_t nnum,
                                                            int32_t e_den, unsigned long long* bad)
{
    const uint32_t m = blockIdx.x * kThreads + threadIdx.x;   // grid covers 2^23 exactly
    const float den = __uint_as_float(((127u + static_cast<uint32_t>(e_den)) << 23) | m);
    uint32_t miss = 0;
    for (int32_t r = 0; r < nnum; ++r) {
        const float num = nums[r];
        miss += same_bits(gemk::div_rn(num, den), num / den) ? 0u : 1u;
    }
    if (miss) atomicAdd(bad, static_cast<unsigned long long>(miss));
}

template <typename Launch>
int run_counting(Launch launch, uint64_t* mismatches)
{
    unsigned long long* d_bad = nullptr;
    if (hipMalloc(&d_bad, sizeof(*d_bad)) != hipSuccess) return GEM_ENOMEM;
    int rc = GEM_OK;
    unsigned long long host = 0;
    if (hipMemset(d_bad, 0, sizeof(*d_bad)) != hipSuccess) rc = GEM_EHIP;
    if (!rc) {
        launch(d_bad);
        if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) rc = GEM_EHIP;
    }
    if (!rc && hipMemcpy(&host, d_bad, sizeof(host), hipMemcpyDeviceToHost) != hipSuccess)
        rc = GEM_EHIP;
    (void)hipFree(d_bad);
    if (!rc) *mismatches = host;
    return rc;
}

}  // namespace

extern "C" {

int gem_selftest_ln_div(uint64_t* mismatches)
{
    if (!mismatches) return GEM_EINVAL;
    return run_counting([](unsigned long long* bad) {
        hipLaunchKernelGGL(ln_div_kernel, dim3((1u << 24) / kThreads), dim3(kThreads), 0, 0, bad);
    }, mismatches);
}

int gem_selftest_radius(uint64_t* mismatches)
{
    if (!mismatches) return GEM_EINVAL;
    return run_counting([](unsigned long long* bad) {
        hipLaunchKernelGGL(radius_kernel, dim3((1u << 24) / kThreads), dim3(kThreads), 0, 0, bad);
    }, mismatches);
}

int gem_selftest_div_random(uint64_t seed, int64_t count, uint64_t* mismatches)
{
    if (!mismatches || count < 0 || count > (int64_t{1} << 34)) return GEM_EINVAL;
    if (count == 0) {
        *mismatches = 0;
        return GEM_OK;
    }
    const unsigned grid = static_cast<unsigned>((count + kThreads - 1) / kThreads);
    return run_counting([&](unsigned long long* bad) {
        hipLaunchKernelGGL(div_random_kernel, dim3(grid), dim3(kThreads), 0, 0, seed, count, bad);
    }, mismatches);
}

// nums: host array of nnum numerators (1 <= nnum <= 4096); e_den in [-126, 127].
int gem_selftest_div_grid(const float* nums, int32_t nnum, int32_t e_den, uint64_t* mismatches)
{
    if (!mismatches || !nums || nnum < 1 || nnum > 4096 || e_den < -126 || e_den > 127)
        return GEM_EINVAL;
    float* d_nums = nullptr;
    if (hipMalloc(&d_nums, sizeof(float) * static_cast<size_t>(nnum)) != hipSuccess) return GEM_ENOMEM;
    int rc = GEM_OK;
    if (hipMemcpy(d_nums, nums, sizeof(float) * static_cast<size_t>(nnum), hipMemcpyHostToDevice) !=
        hipSuccess)
        rc = GEM_EHIP;
    if (!rc)
        rc = run_counting([&](unsigned long long* bad) {
            hipLaunchKernelGGL(div_grid_kernel, dim3((1u << 23) / kThreads), dim3(kThreads), 0, 0,
                               d_nums, nnum, e_den, bad);
        }, mismatches);
    (void)hipFree(d_nums);
    return rc;
}

}  // extern "C"

// bdlm_probe.hip -- measurement only, not part of libbdlm: a plain streaming kernel with
// the byte shape of a block-step launch, built into libbdlm_probe.so for the benchmark.
//
// Per unit (one (batch row, head) of a block step) it reads an input slab and a state
// slab and writes an output slab, with the access pattern a bandwidth-bound kernel
// would use on gfx950 (16-byte vector loads, nontemporal or not, several in flight per
// lane, 16-byte stores; the small input slab first, which measured faster than state
// first) and no arithmetic beyond folding the loaded values into what it stores.  The time of a launch over the same bytes as a block step is the ceiling a
// launch of that size reaches here; the benchmark reports it beside the step.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Workgroup `split * unit + part` streams part `part` of unit `unit`'s three slabs.
// Slab sizes are in 16-byte vectors and divisible by split (checked on the host).
template <bool NT>
__device__ __forceinline__ f32x4 ld(const f32x4 *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}
template <int TPB, int UNR, bool NT>
__global__ void __launch_bounds__(TPB) probe_kernel(const f32x4 *st, const f32x4 *in, f32x4 *out,
                                                    int64_t st_n, int64_t in_n, int64_t out_n,
                                                    int split) {
    const int64_t unit = blockIdx.x / split, part = blockIdx.x % split;
    const int64_t sn = st_n / split, qn = in_n / split, on = out_n / split;
    const f32x4 *s = st + unit * st_n + part * sn;
    const f32x4 *q = in + unit * in_n + part * qn;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t i = threadIdx.x; i < qn; i += TPB) acc += ld<NT>(q + i);
    for (int64_t i0 = threadIdx.x; i0 < sn; i0 += TPB * UNR) {
        f32x4 v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t i = i0 + u * TPB;
            v[u] = i < sn ? ld<NT>(s + i) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) acc += v[u];
    }
    f32x4 *o = out + unit * out_n + part * on;
    for (int64_t i = threadIdx.x; i < on; i += TPB) {
        if constexpr (NT) __builtin_nontemporal_store(acc, o + i);
        else o[i] = acc;
    }
}

}  // namespace

extern "C" {

// Launch configurations the probe offers (the benchmark keeps the fastest): threads per
// workgroup, workgroups per unit, nontemporal or not.
static const int kSplit[] = {1, 2, 4, 1, 2, 4, 2, 1, 2};
static const int kTpb[] = {256, 256, 256, 512, 512, 512, 1024, 256, 256};
static const int kNt[] = {1, 1, 1, 1, 1, 1, 1, 0, 0};
static const int kNcfg = sizeof(kSplit) / sizeof(kSplit[0]);
int bdlm_probe_configs(void) { return kNcfg; }

// Enqueue one probe launch: `units` units of st_bytes / in_bytes / out_bytes each
// (multiples of 16 * split), launch configuration `cfg` (0 .. bdlm_probe_configs() - 1):
// threads per workgroup and workgroups per unit.  Device pointers, 16-byte aligned.
// Returns 0, or -1 for a bad argument, -2 if the launch failed.
int bdlm_probe_stream(const void *st, const void *in, void *out, int64_t units, int64_t st_bytes,
                      int64_t in_bytes, int64_t out_bytes, int cfg, void *stream) {
    if (cfg < 0 || cfg >= kNcfg || units <= 0 || !st || !in || !out) return -1;
    const int split = kSplit[cfg];
    const int64_t q = 16 * split;
    if (st_bytes % q || in_bytes % q || out_bytes % q || units * split > (int64_t(1) << 30)) return -1;
    const dim3 grid(static_cast<unsigned>(units * split));
    hipStream_t s = static_cast<hipStream_t>(stream);
    const f32x4 *S = static_cast<const f32x4 *>(st), *I = static_cast<const f32x4 *>(in);
    f32x4 *O = static_cast<f32x4 *>(out);
    const int64_t sn = st_bytes / 16, in_n = in_bytes / 16, on = out_bytes / 16;
    if (!kNt[cfg])
        hipLaunchKernelGGL((probe_kernel<256, 8, false>), grid, dim3(256), 0, s, S, I, O, sn, in_n, on,
                           split);
    else if (kTpb[cfg] == 256)
        hipLaunchKernelGGL((probe_kernel<256, 8, true>), grid, dim3(256), 0, s, S, I, O, sn, in_n, on,
                           split);
    else if (kTpb[cfg] == 512)
        hipLaunchKernelGGL((probe_kernel<512, 4, true>), grid, dim3(512), 0, s, S, I, O, sn, in_n, on,
                           split);
    else
        hipLaunchKernelGGL((probe_kernel<1024, 2, true>), grid, dim3(1024), 0, s, S, I, O, sn, in_n,
                           on, split);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"

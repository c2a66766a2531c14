// Compacted prompt cache (Appendix B: retained tokens in temporal order,
// inserted through the standard cache update) on gfx950: a pure byte copy.
// Sixteen consecutive threads move one 256-byte row in 16-byte vectors, so
// a wave streams four rows per instruction with fully coalesced stores.
#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr int kGatherThreads = 256;

__global__ void __launch_bounds__(kGatherThreads) gather_kernel(GatherArgs a) {
    const int c = blockIdx.y, b = blockIdx.z;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int vec_per_row = a.row_bytes / 16;
    const int64_t item = static_cast<int64_t>(blockIdx.x) * kGatherThreads + threadIdx.x;
    const int j = static_cast<int>(item / vec_per_row);
    const int q = static_cast<int>(item - static_cast<int64_t>(j) * vec_per_row);
    if (j >= a.c_max) return;
    const int n = a.counts[hc];
    const int t = (j < n) ? a.idx[hc * a.c_max + j] : -1;
    const bool ok = t >= 0 && t < a.T;
    uint4 kv = make_uint4(0u, 0u, 0u, 0u), vv = kv;
    if (ok) {
        const char* ks = static_cast<const char*>(a.k) +
                         (static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                          static_cast<int64_t>(t) * a.kst) * a.elem_bytes;
        const char* vs = static_cast<const char*>(a.v) +
                         (static_cast<int64_t>(b) * a.vsb + static_cast<int64_t>(c) * a.vsh +
                          static_cast<int64_t>(t) * a.vst) * a.elem_bytes;
        kv = *reinterpret_cast<const uint4*>(ks + 16 * q);
        vv = *reinterpret_cast<const uint4*>(vs + 16 * q);
    }
    const int64_t o = (hc * a.c_max + j) * static_cast<int64_t>(a.row_bytes) + 16 * q;
    *reinterpret_cast<uint4*>(static_cast<char*>(a.k_out) + o) = kv;
    *reinterpret_cast<uint4*>(static_cast<char*>(a.v_out) + o) = vv;
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
    const int64_t items = static_cast<int64_t>(a.c_max) * (a.row_bytes / 16);
    dim3 grid(static_cast<unsigned>((items + kGatherThreads - 1) / kGatherThreads), a.Hkv, a.B);
    hipLaunchKernelGGL(gather_kernel, grid, dim3(kGatherThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace mmskv

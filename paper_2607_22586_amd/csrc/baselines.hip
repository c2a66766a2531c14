// Baseline selectors on the same scoring and selection kernels: the comparison
// methods as the paper configures them (SnapKV, StreamingLLM, ExpectedAttn).
// Each reduces to a per-key score for the MASS-mode top-C:
//   window_rows_kernel   the last n window queries of each head in the form of
//                        proxies (scaled by log2(e)/sqrt(d), bf16) -- SnapKV's
//                        observation window, scored by the mass pass;
//   shape_scores_kernel  SnapKV: average pooling of the masses over the keys
//                        before the window, the window kept; StreamingLLM:
//                        sinks kept, then recency; sinks only: the masses with
//                        the first keys kept.  A kept key scores 2^100.
#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr float kKeepScore = 0x1p100f;

__global__ void __launch_bounds__(256) window_rows_kernel(WindowArgs a) {
    const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t total = static_cast<int64_t>(a.B) * a.Hq * a.n * a.d;
    if (e >= total) return;
    const int j = static_cast<int>(e % a.d);
    const int64_t rowi = e / a.d;                     // (b, h, i)
    const int i = static_cast<int>(rowi % a.n);
    const int64_t bh = rowi / a.n;
    const int h = static_cast<int>(bh % a.Hq), b = static_cast<int>(bh / a.Hq);
    const int w = a.W - a.n + i;
    const int64_t off = static_cast<int64_t>(b) * a.qsb + static_cast<int64_t>(h) * a.qsh +
                        static_cast<int64_t>(w) * a.qst + j;
    // the window query as a bf16 value (fp32 inputs rounded to nearest even)
    const uint32_t qb = a.q_dtype == 1 ? static_cast<uint32_t>(static_cast<const uint16_t*>(a.q)[off])
                                       : f32_to_bf16_bits(static_cast<const float*>(a.q)[off]);
    const double v = static_cast<double>(__uint_as_float(qb << 16)) * a.scale;
    a.rows[rowi * a.d + j] = static_cast<uint16_t>(f32_to_bf16_bits(static_cast<float>(v)));
    if (w == a.W - 1) a.q_last[bh * a.d + j] = static_cast<uint16_t>(qb);
}

__global__ void __launch_bounds__(256) shape_scores_kernel(ShapeArgs a) {
    const int t = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
    const int64_t bc = blockIdx.y;
    if (t >= a.T) return;
    const float* m = a.mass + bc * a.T;
    float s;
    if (a.kind == 0) {                                // SnapKV
        const int prefix = a.T - a.window;
        if (t >= prefix) {
            s = kKeepScore;
        } else {
            float sum = 0.f;
            for (int u = t - a.pool / 2; u <= t + a.pool / 2; ++u)
                if (u >= 0 && u < prefix) sum += m[u];
            s = sum / static_cast<float>(a.pool);
        }
    } else if (a.kind == 1) {                         // StreamingLLM
        s = t < a.sinks ? kKeepScore : static_cast<float>(t);
    } else {                                          // sinks only
        s = t < a.sinks ? kKeepScore : m[t];
    }
    a.score[bc * a.T + t] = s;
}

}  // namespace

hipError_t launch_window_rows(const WindowArgs& a, hipStream_t s) {
    const int64_t total = static_cast<int64_t>(a.B) * a.Hq * a.n * a.d;
    hipLaunchKernelGGL(window_rows_kernel, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_shape_scores(const ShapeArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(shape_scores_kernel, dim3((a.T + 255) / 256, a.B * a.Hkv), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace mmskv

// C ABI of libmmshiftkv: argument validation, workspace sizing and kernel
// launches.  Every check runs on the host before anything is enqueued.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "../../include/mmshiftkv.h"
#include "kernels.hpp"

using namespace mmskv;

namespace {

// Softmax scale carried by the queries (Sec. 3.2.2 Eq. 7's 1/sqrt(d), with
// log2(e) so that the products are base-2 logits), in fp64: the proxies are
// multiplied by it before their bf16 rounding and the score passes apply it
// to the anchor rows the same way.
double query_scale(int d) { return 1.4426950408889634074 / sqrt(static_cast<double>(d)); }


constexpr size_t kAlign = 256;
constexpr size_t kMaxRowLds = 96 * 1024;   // Gh * P + 32 rows of fp32 in LDS
constexpr size_t kMaxRowLds8 = 64 * 1024;  // the same with 8-wave mass blocks

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

int elem_bytes(int32_t dtype) { return dtype == MMSKV_F32 ? 4 : (dtype == MMSKV_BF16 ? 2 : 0); }

// The head layout every call reads: B, Hq, Hkv (Hq % Hkv == 0) and T.
int check_heads(const mmskv_shape* s) {
    if (s == nullptr) return MMSKV_EINVAL;
    if (s->B < 1 || s->B > 65535 || s->Hq < 1 || s->Hkv < 1 || s->Hkv > 65535 || s->T < 1) return MMSKV_EINVAL;
    if (s->Hq % s->Hkv != 0) return MMSKV_EINVAL;
    return MMSKV_OK;
}

// The whole shape, for the calls that read the window queries and scores.
int check_shape(const mmskv_shape* s) {
    int rc = check_heads(s);
    if (rc) return rc;
    if (s->W < 1 || s->d < 1) return MMSKV_EINVAL;
    if (s->d != 64 && s->d != 128) return MMSKV_EUNSUPPORTED;
    return MMSKV_OK;
}

// The parameters that the selection reads (group layout, tau, lambda, mode).
int check_method(const mmskv_params* p) {
    if (p == nullptr) return MMSKV_EINVAL;
    if (p->P < 1 || p->G < 1 || p->P % p->G != 0) return MMSKV_EINVAL;
    if (p->G > 255) return MMSKV_EUNSUPPORTED;
    if ((p->P / p->G) % 16 != 0 || p->P % 32 != 0) return MMSKV_EUNSUPPORTED;
    if (!(p->tau > 0.0 && p->tau <= 1.0)) return MMSKV_EINVAL;
    if (!(p->lambda >= 0.0) || !isfinite(p->lambda)) return MMSKV_EINVAL;
    if (p->mode != MMSKV_VOTE && p->mode != MMSKV_MASS) return MMSKV_EINVAL;
    if (p->keep_last != 0 && p->keep_last != 1) return MMSKV_EINVAL;
    return MMSKV_OK;
}

// Every parameter (the proxy and score calls).
int check_params(const mmskv_shape* s, const mmskv_params* p) {
    int rc = check_method(p);
    if (rc) return rc;
    if (!(p->gamma >= 0.0) || !isfinite(p->gamma)) return MMSKV_EINVAL;
    if (p->std_ddof != 0 && p->std_ddof != 1) return MMSKV_EINVAL;
    if (s->W - p->std_ddof < 1) return MMSKV_EINVAL;
    if (p->layer < 0 || p->layer > 65535) return MMSKV_EINVAL;
    return MMSKV_OK;
}

int check_rows(const void* base, const mmskv_strides* st, int eb, bool vec16) {
    if (st == nullptr) return MMSKV_EINVAL;
    if (st->sb < 0 || st->sh < 0 || st->st < 0) return MMSKV_EINVAL;
    if (vec16) {
        if (!aligned(base, 16)) return MMSKV_EINVAL;
        if ((st->sb * eb) % 16 || (st->sh * eb) % 16 || (st->st * eb) % 16) return MMSKV_EINVAL;
    } else if (!aligned(base, static_cast<size_t>(eb))) {
        return MMSKV_EINVAL;
    }
    return MMSKV_OK;
}

int status_of(hipError_t e) { return e == hipSuccess ? MMSKV_OK : MMSKV_EHIP; }

struct ScoreLayout {
    ScorePlan plan;
    int n_kb, block_keys, mass_n_kb, rows, rows_pad;
    size_t part_bytes, lse_off, total;
};

ScoreLayout score_layout(const mmskv_shape* s, const mmskv_params* p) {
    ScoreLayout l;
    const int Gh = s->Hq / s->Hkv;
    l.plan = score_plan(s->B, s->Hkv, s->T);
    const int lse_keys = 32 * l.plan.lse_sub * l.plan.lse_waves;
    l.n_kb = (s->T + lse_keys - 1) / lse_keys;
    l.block_keys = 64 * l.plan.mass_waves;
    l.mass_n_kb = (s->T + l.block_keys - 1) / l.block_keys;
    l.rows = Gh * p->P;
    l.rows_pad = l.rows + 32 * ((Gh + 31) / 32);
    // 8-wave mass blocks hold 8 staged tiles (68 KiB at d = 128) next to the
    // row normalisers; many rows take 4-wave blocks, which stage 4
    if (l.plan.mass_waves == 8 && static_cast<size_t>(l.rows_pad) * sizeof(float) > kMaxRowLds8) {
        l.plan.mass_waves = 4;
        l.block_keys = 64 * l.plan.mass_waves;
        l.mass_n_kb = (s->T + l.block_keys - 1) / l.block_keys;
    }
    const size_t heads = static_cast<size_t>(s->B) * s->Hkv;
    l.part_bytes = heads * l.n_kb * l.rows_pad * sizeof(float2);
    l.lse_off = align_up(l.part_bytes);
    l.total = l.lse_off + align_up(heads * l.rows_pad * sizeof(float));
    return l;
}

struct SelectLayout {
    size_t theta_off, tcut_off, keys_off, planes_off, hist_off, total;
};

SelectLayout select_layout(const mmskv_shape* s, const mmskv_params* p) {
    SelectLayout l;
    const size_t heads = static_cast<size_t>(s->B) * s->Hkv;
    l.theta_off = 0;
    l.tcut_off = align_up(heads * p->G * sizeof(uint32_t));
    l.keys_off = l.tcut_off + align_up(heads * p->G * sizeof(int32_t));
    l.planes_off = l.keys_off + align_up(heads * static_cast<size_t>(select_key_stride(s->T)) * sizeof(uint64_t));
    const size_t words = (static_cast<size_t>(s->T) + 31) / 32;
    l.hist_off = l.planes_off + align_up(heads * words * p->G * sizeof(uint32_t));
    l.total = l.hist_off + align_up(heads * 2048 * sizeof(uint32_t));
    return l;
}

// Shared validation and argument packing of the three score entry points.
int prepare_score(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                  const uint16_t* q_last, const void* k, int32_t k_dtype,
                  const mmskv_strides* k_strides, void* ws, size_t ws_bytes, ScoreArgs* a) {
    int rc = check_shape(shape);
    if (rc) return rc;
    rc = check_params(shape, params);
    if (rc) return rc;
    const int eb = elem_bytes(k_dtype);
    if (eb == 0) return MMSKV_EINVAL;
    if (proxies == nullptr || q_last == nullptr || k == nullptr) return MMSKV_EINVAL;
    if (!aligned(proxies, 16) || !aligned(q_last, 16)) return MMSKV_EINVAL;
    rc = check_rows(k, k_strides, eb, true);
    if (rc) return rc;
    const ScoreLayout l = score_layout(shape, params);
    // the mass pass keeps one head's row normalisers (rows_pad floats) in LDS
    if (static_cast<size_t>(l.rows_pad) * sizeof(float) > kMaxRowLds) return MMSKV_EUNSUPPORTED;
    if (ws == nullptr || !aligned(ws, kAlign) || ws_bytes < l.total) return MMSKV_EWORKSPACE;
    a->proxies = proxies;
    a->q_last = q_last;
    a->k = k;
    a->k_dtype = k_dtype;
    a->ksb = k_strides->sb;
    a->ksh = k_strides->sh;
    a->kst = k_strides->st;
    a->B = shape->B;
    a->Hq = shape->Hq;
    a->Hkv = shape->Hkv;
    a->T = shape->T;
    a->d = shape->d;
    a->P = params->P;
    a->G = params->G;
    a->Gh = shape->Hq / shape->Hkv;
    a->lse_waves = l.plan.lse_waves;
    a->lse_sub = l.plan.lse_sub;
    a->n_kb = l.n_kb;
    a->block_keys = l.block_keys;
    a->mass_n_kb = l.mass_n_kb;
    a->rows = l.rows;
    a->rows_pad = l.rows_pad;
    a->anchor_scale = query_scale(shape->d);
    a->lane_sum_hi = lane_sum_limit(shape->T, 16);     // pass 1 sums 16 keys per lane and chain
    a->part = static_cast<float2*>(ws);
    a->lse = reinterpret_cast<float*>(static_cast<char*>(ws) + l.lse_off);
    a->group_mass = nullptr;
    a->mass = nullptr;
    a->anchor = nullptr;
    return MMSKV_OK;
}

int check_score_outputs(const mmskv_params* p, const float* gm, const float* mass, const float* an) {
    if (mass == nullptr || an == nullptr) return MMSKV_EINVAL;
    if (p->mode == MMSKV_VOTE && gm == nullptr) return MMSKV_EINVAL;
    if (!aligned(mass, 4) || !aligned(an, 4) || (gm && !aligned(gm, 4))) return MMSKV_EINVAL;
    return MMSKV_OK;
}

constexpr int kHiddenChunk = 256;   // tokens per partial sum of the hidden statistics

int check_hshape(const mmskv_hshape* s) {
    if (s == nullptr) return MMSKV_EINVAL;
    if (s->B < 1 || s->B > 65535 || s->T < 1 || s->D < 8 || s->D % 8 != 0) return MMSKV_EINVAL;
    return MMSKV_OK;
}

size_t hidden_stats_ws(const mmskv_hshape* s) {
    const size_t chunks = (static_cast<size_t>(s->T) + kHiddenChunk - 1) / kHiddenChunk;
    return align_up(static_cast<size_t>(s->B) * chunks * s->D * sizeof(double2));
}

}  // namespace

extern "C" {

int mmshiftkv_version(void) { return 100; }

const char* mmshiftkv_status_string(int status) {
    switch (status) {
        case MMSKV_OK: return "ok";
        case MMSKV_EINVAL: return "invalid argument";
        case MMSKV_EUNSUPPORTED: return "unsupported configuration";
        case MMSKV_EWORKSPACE: return "workspace missing, misaligned or too small";
        case MMSKV_EHIP: return "HIP launch error";
        case MMSKV_ESCRATCH: return "problem needs more scratch memory than the allocation-free entry point holds";
        default: return "unknown status";
    }
}

int mmshiftkv_build_proxies(const mmskv_shape* shape, const mmskv_params* params, const void* q_win,
                            int32_t q_dtype, const mmskv_strides* q_strides, const float* rope_cos_f,
                            const float* rope_sin_f, const float* rope_cos_l, const float* rope_sin_l,
                            uint16_t* proxies, uint16_t* q_last, double* stats, void* stream) {
    int rc = check_shape(shape);
    if (rc) return rc;
    rc = check_params(shape, params);
    if (rc) return rc;
    const int eb = elem_bytes(q_dtype);
    if (eb == 0 || q_win == nullptr || proxies == nullptr || q_last == nullptr) return MMSKV_EINVAL;
    rc = check_rows(q_win, q_strides, eb, false);
    if (rc) return rc;
    if ((rope_cos_f == nullptr) != (rope_sin_f == nullptr)) return MMSKV_EINVAL;
    if ((rope_cos_l == nullptr) != (rope_sin_l == nullptr)) return MMSKV_EINVAL;
    if (!aligned(proxies, 8) || !aligned(q_last, 2) || (stats && !aligned(stats, 8))) return MMSKV_EINVAL;
    ProxyArgs a;
    a.q = q_win;
    a.q_dtype = q_dtype;
    a.qsb = q_strides->sb;
    a.qsh = q_strides->sh;
    a.qst = q_strides->st;
    a.cos_f = rope_cos_f;
    a.sin_f = rope_sin_f;
    a.cos_l = rope_cos_l;
    a.sin_l = rope_sin_l;
    a.proxies = proxies;
    a.q_last = q_last;
    a.stats = stats;
    a.B = shape->B;
    a.Hq = shape->Hq;
    a.W = shape->W;
    a.d = shape->d;
    a.P = params->P;
    a.ddof = params->std_ddof;
    a.layer = params->layer;
    a.gamma = params->gamma;
    a.scale = query_scale(shape->d);
    a.key0 = static_cast<uint32_t>(params->seed & 0xFFFFFFFFull);
    a.key1 = static_cast<uint32_t>(params->seed >> 32);
    return status_of(launch_build_proxies(a, static_cast<hipStream_t>(stream)));
}

size_t mmshiftkv_score_workspace(const mmskv_shape* shape, const mmskv_params* params) {
    if (check_shape(shape) || check_params(shape, params)) return 0;
    return score_layout(shape, params).total;
}

static int score_lse_stages(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                            const uint16_t* q_last, const void* k, int32_t k_dtype,
                            const mmskv_strides* k_strides, void* workspace, size_t workspace_bytes,
                            void* stream, int stages) {
    ScoreArgs a;
    int rc = prepare_score(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace,
                           workspace_bytes, &a);
    if (rc) return rc;
    return status_of(launch_score_lse(a, stages, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_score_lse(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                        const uint16_t* q_last, const void* k, int32_t k_dtype,
                        const mmskv_strides* k_strides, void* workspace, size_t workspace_bytes,
                        void* stream) {
    return score_lse_stages(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace, workspace_bytes,
                            stream, kLseBlocks | kLseMerge);
}

int mmshiftkv_score_lse_blocks(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                               const uint16_t* q_last, const void* k, int32_t k_dtype,
                               const mmskv_strides* k_strides, void* workspace, size_t workspace_bytes,
                               void* stream) {
    return score_lse_stages(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace, workspace_bytes,
                            stream, kLseBlocks);
}

int mmshiftkv_score_lse_merge(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                              const uint16_t* q_last, const void* k, int32_t k_dtype,
                              const mmskv_strides* k_strides, void* workspace, size_t workspace_bytes,
                              void* stream) {
    return score_lse_stages(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace, workspace_bytes,
                            stream, kLseMerge);
}

int mmshiftkv_score_mass(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                         const uint16_t* q_last, const void* k, int32_t k_dtype,
                         const mmskv_strides* k_strides, float* group_mass, float* mass, float* anchor,
                         void* workspace, size_t workspace_bytes, void* stream) {
    ScoreArgs a;
    int rc = prepare_score(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace,
                           workspace_bytes, &a);
    if (rc) return rc;
    rc = check_score_outputs(params, group_mass, mass, anchor);
    if (rc) return rc;
    a.group_mass = group_mass;
    a.mass = mass;
    a.anchor = anchor;
    return status_of(launch_score_mass(a, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_score(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                    const uint16_t* q_last, const void* k, int32_t k_dtype,
                    const mmskv_strides* k_strides, float* group_mass, float* mass, float* anchor,
                    void* workspace, size_t workspace_bytes, void* stream) {
    ScoreArgs a;
    int rc = prepare_score(shape, params, proxies, q_last, k, k_dtype, k_strides, workspace,
                           workspace_bytes, &a);
    if (rc) return rc;
    rc = check_score_outputs(params, group_mass, mass, anchor);
    if (rc) return rc;
    a.group_mass = group_mass;
    a.mass = mass;
    a.anchor = anchor;
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = status_of(launch_score_lse(a, kLseBlocks | kLseMerge, s));
    if (rc) return rc;
    return status_of(launch_score_mass(a, s));
}

}  // extern "C"

namespace {

// Scratch memory of mmshiftkv_score_noalloc: one array per GPU, held until
// the process ends.  In host code `scratch` names a host-side stand-in, so
// the device address of each GPU's copy is taken once, with that GPU
// current, and only that address is handed to the kernels.
constexpr size_t kScratchBytes = MMSKV_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MMSKV_EHIP;
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return MMSKV_EHIP;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return MMSKV_OK;
}

}  // namespace

extern "C" {

int mmshiftkv_score_noalloc(const mmskv_shape* shape, const mmskv_params* params, const uint16_t* proxies,
                            const uint16_t* q_last, const void* k, int32_t k_dtype,
                            const mmskv_strides* k_strides, float* group_mass, float* mass, float* anchor,
                            void* stream) {
    int rc = check_shape(shape);
    if (rc) return rc;
    rc = check_params(shape, params);
    if (rc) return rc;
    if (score_layout(shape, params).total > kScratchBytes) return MMSKV_ESCRATCH;
    void* ws = nullptr;
    rc = scratch_address(&ws);
    if (rc) return rc;
    // every byte of the workspace that the passes read is written first by
    // the same call, so nothing needs clearing
    return mmshiftkv_score(shape, params, proxies, q_last, k, k_dtype, k_strides, group_mass, mass, anchor, ws,
                           kScratchBytes, stream);
}

size_t mmshiftkv_select_workspace(const mmskv_shape* shape, const mmskv_params* params) {
    if (check_heads(shape) || check_method(params)) return 0;
    return select_layout(shape, params).total;
}

namespace {

// Validation and argument packing of the selection calls; `stages` is a mask
// of kSelectTau, kSelectVote, kSelectPick, each stage checking the
// arguments it reads.
int select_call(const mmskv_shape* shape, const mmskv_params* params, const float* group_mass, const float* mass,
                const float* anchor, const int32_t* budgets, int32_t budget, int32_t c_max, int32_t* idx,
                int32_t* counts, uint8_t* votes, void* workspace, size_t workspace_bytes, void* stream, int stages) {
    int rc = check_heads(shape);
    if (rc) return rc;
    rc = check_method(params);
    if (rc) return rc;
    const bool vote = params->mode == MMSKV_VOTE;
    if ((stages & kSelectTau) && vote && group_mass == nullptr) return MMSKV_EINVAL;
    if (stages & kSelectVote) {
        if (vote && anchor == nullptr) return MMSKV_EINVAL;
        if (!vote && (mass == nullptr || votes != nullptr)) return MMSKV_EINVAL;
    }
    if (stages & kSelectPick) {
        if (idx == nullptr || counts == nullptr || c_max < 1) return MMSKV_EINVAL;
        if (budgets == nullptr && (budget < 1 || c_max < (budget < shape->T ? budget : shape->T)))
            return MMSKV_EINVAL;
    }
    const SelectLayout l = select_layout(shape, params);
    if (workspace == nullptr || !aligned(workspace, kAlign) || workspace_bytes < l.total)
        return MMSKV_EWORKSPACE;
    SelectArgs a;
    a.group_mass = group_mass;
    a.mass = mass;
    a.anchor = anchor;
    a.budgets = budgets;
    a.B = shape->B;
    a.Hkv = shape->Hkv;
    a.T = shape->T;
    a.G = params->G;
    a.mode = params->mode;
    a.keep_last = params->keep_last;
    a.budget = budget;
    a.c_max = c_max;
    a.tau = params->tau;
    a.lambda = params->lambda;
    // fixed-point unit 2^-S with S = 62 - bitlen(rows per group), so a
    // group's total (<= rows per group, plus rounding) stays below 2^63
    {
        const int rows_per_group = (params->P / params->G) * (shape->Hq / shape->Hkv);
        int bits = 0;
        while ((1 << bits) <= rows_per_group) ++bits;
        a.fix_shift = 62 - bits;
    }
    char* w = static_cast<char*>(workspace);
    a.theta = reinterpret_cast<uint32_t*>(w + l.theta_off);
    a.tcut = reinterpret_cast<int32_t*>(w + l.tcut_off);
    a.keys = reinterpret_cast<uint64_t*>(w + l.keys_off);
    a.planes = reinterpret_cast<uint32_t*>(w + l.planes_off);
    a.hist0 = reinterpret_cast<uint32_t*>(w + l.hist_off);
    a.kpt = select_kpt(shape->T);
    a.key_stride = select_key_stride(shape->T);
    a.idx = idx;
    a.counts = counts;
    a.votes = votes;
    return status_of(launch_select(a, stages, static_cast<hipStream_t>(stream)));
}

}  // namespace

int mmshiftkv_select_topk(const mmskv_shape* shape, const mmskv_params* params, const float* group_mass,
                          const float* mass, const float* anchor, const int32_t* budgets, int32_t budget,
                          int32_t c_max, int32_t* idx, int32_t* counts, uint8_t* votes, void* workspace,
                          size_t workspace_bytes, void* stream) {
    return select_call(shape, params, group_mass, mass, anchor, budgets, budget, c_max, idx, counts, votes,
                       workspace, workspace_bytes, stream, kSelectTau | kSelectVote | kSelectPick);
}

int mmshiftkv_select_tau(const mmskv_shape* shape, const mmskv_params* params, const float* group_mass,
                         void* workspace, size_t workspace_bytes, void* stream) {
    return select_call(shape, params, group_mass, nullptr, nullptr, nullptr, 0, 0, nullptr, nullptr, nullptr,
                       workspace, workspace_bytes, stream, kSelectTau);
}

int mmshiftkv_select_vote(const mmskv_shape* shape, const mmskv_params* params, const float* mass,
                          const float* anchor, uint8_t* votes, void* workspace, size_t workspace_bytes,
                          void* stream) {
    return select_call(shape, params, nullptr, mass, anchor, nullptr, 0, 0, nullptr, nullptr, votes, workspace,
                       workspace_bytes, stream, kSelectVote);
}

int mmshiftkv_select_pick(const mmskv_shape* shape, const mmskv_params* params, const int32_t* budgets,
                          int32_t budget, int32_t c_max, int32_t* idx, int32_t* counts, void* workspace,
                          size_t workspace_bytes, void* stream) {
    return select_call(shape, params, nullptr, nullptr, nullptr, budgets, budget, c_max, idx, counts, nullptr,
                       workspace, workspace_bytes, stream, kSelectPick);
}

int mmshiftkv_gather_kv(const mmskv_shape* shape, const void* k, const void* v, int32_t dtype,
                        const mmskv_strides* k_strides, const mmskv_strides* v_strides,
                        const int32_t* idx, const int32_t* counts, int32_t c_max, void* k_out,
                        void* v_out, void* stream) {
    if (shape == nullptr) return MMSKV_EINVAL;
    if (shape->B < 1 || shape->B > 65535 || shape->Hkv < 1 || shape->Hkv > 65535 || shape->T < 1 ||
        shape->d < 1 || shape->d > 65536)
        return MMSKV_EINVAL;
    const int eb = elem_bytes(dtype);
    if (eb == 0 || (shape->d * eb) % 16 != 0) return MMSKV_EINVAL;
    if (k == nullptr || v == nullptr || idx == nullptr || counts == nullptr || c_max < 1 || k_out == nullptr ||
        v_out == nullptr)
        return MMSKV_EINVAL;
    int rc = check_rows(k, k_strides, eb, true);
    if (rc) return rc;
    rc = check_rows(v, v_strides, eb, true);
    if (rc) return rc;
    if (!aligned(k_out, 16) || !aligned(v_out, 16)) return MMSKV_EINVAL;
    GatherArgs a;
    a.k = k;
    a.v = v;
    a.ksb = k_strides->sb;
    a.ksh = k_strides->sh;
    a.kst = k_strides->st;
    a.vsb = v_strides->sb;
    a.vsh = v_strides->sh;
    a.vst = v_strides->st;
    a.elem_bytes = eb;
    a.row_bytes = shape->d * eb;
    a.idx = idx;
    a.counts = counts;
    a.B = shape->B;
    a.Hkv = shape->Hkv;
    a.T = shape->T;
    a.c_max = c_max;
    a.k_out = k_out;
    a.v_out = v_out;
    return status_of(launch_gather(a, static_cast<hipStream_t>(stream)));
}

namespace {

int check_decode(const mmskv_shape* shape, int32_t n_dec) {
    int rc = check_shape(shape);
    if (rc) return rc;
    if (n_dec < 1) return MMSKV_EINVAL;
    const int64_t rows = static_cast<int64_t>(shape->Hq / shape->Hkv) * n_dec;
    if (rows > decode_max_rows()) return MMSKV_EUNSUPPORTED;
    return MMSKV_OK;
}

// partials, then the scaled decode queries
size_t decode_part_bytes(const mmskv_shape* shape, int32_t n_dec) {
    const int64_t Gh = shape->Hq / shape->Hkv;
    return align_up(static_cast<size_t>(shape->B) * shape->Hkv * decode_key_blocks(shape->T) *
                    decode_rows_pad(static_cast<int>(Gh), n_dec) * sizeof(float4));
}

size_t decode_ws(const mmskv_shape* shape, int32_t n_dec) {
    const int64_t Gh = shape->Hq / shape->Hkv;
    return decode_part_bytes(shape, n_dec) +
           align_up(static_cast<size_t>(shape->B) * shape->Hkv * decode_rows_pad(static_cast<int>(Gh), n_dec) *
                    shape->d * sizeof(uint16_t));
}

}  // namespace

size_t mmshiftkv_decode_workspace(const mmskv_shape* shape, int32_t n_dec) {
    if (check_decode(shape, n_dec) != MMSKV_OK) return 0;
    return decode_ws(shape, n_dec);
}

int mmshiftkv_decode_check(const mmskv_shape* shape, int32_t n_dec, const uint16_t* q_dec, const void* k,
                           int32_t dtype, const mmskv_strides* k_strides, const int32_t* idx,
                           const int32_t* counts, int32_t c_max, const void* k_out, const void* v_out,
                           float* coverage, float* out, void* workspace, size_t workspace_bytes,
                           void* stream) {
    int rc = check_decode(shape, n_dec);
    if (rc) return rc;
    const int eb = elem_bytes(dtype);
    if (eb == 0 || q_dec == nullptr || k == nullptr || idx == nullptr || counts == nullptr ||
        k_out == nullptr || v_out == nullptr || coverage == nullptr || out == nullptr)
        return MMSKV_EINVAL;
    if (c_max < 1) return MMSKV_EINVAL;
    if (c_max > decode_max_compact()) return MMSKV_EUNSUPPORTED;
    rc = check_rows(k, k_strides, eb, true);
    if (rc) return rc;
    if (!aligned(q_dec, 16) || !aligned(k_out, 16) || !aligned(v_out, 16) || !aligned(idx, 4) ||
        !aligned(counts, 4) || !aligned(coverage, 4) || !aligned(out, 4))
        return MMSKV_EINVAL;
    if (workspace == nullptr || !aligned(workspace, kAlign) || workspace_bytes < decode_ws(shape, n_dec))
        return MMSKV_EWORKSPACE;
    DecodeArgs a = {};
    a.q_dec = q_dec;
    a.k = k;
    a.k_dtype = dtype;
    a.ksb = k_strides->sb;
    a.ksh = k_strides->sh;
    a.kst = k_strides->st;
    a.idx = idx;
    a.counts = counts;
    a.k_out = k_out;
    a.v_out = v_out;
    a.B = shape->B;
    a.Hq = shape->Hq;
    a.Hkv = shape->Hkv;
    a.T = shape->T;
    a.d = shape->d;
    a.Gh = shape->Hq / shape->Hkv;
    a.n_dec = n_dec;
    a.c_max = c_max;
    a.rows = a.Gh * n_dec;
    a.rows_pad = decode_rows_pad(a.Gh, n_dec);
    a.n_kb = decode_key_blocks(shape->T);
    a.scale = query_scale(shape->d);
    a.lane_sum_hi = lane_sum_limit(shape->T, 32);
    a.part = static_cast<float4*>(workspace);
    a.qsc = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + decode_part_bytes(shape, n_dec));
    a.coverage = coverage;
    a.out = out;
    return status_of(launch_decode_check(a, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_window_rows(const mmskv_shape* shape, int32_t n, const void* q_win, int32_t q_dtype,
                          const mmskv_strides* q_strides, uint16_t* rows, uint16_t* q_last, void* stream) {
    int rc = check_shape(shape);
    if (rc) return rc;
    const int eb = elem_bytes(q_dtype);
    if (eb == 0 || q_win == nullptr || rows == nullptr || q_last == nullptr) return MMSKV_EINVAL;
    if (n < 1 || n > shape->W) return MMSKV_EINVAL;
    rc = check_rows(q_win, q_strides, eb, false);
    if (rc) return rc;
    if (!aligned(rows, 2) || !aligned(q_last, 2)) return MMSKV_EINVAL;
    WindowArgs a;
    a.q = q_win;
    a.q_dtype = q_dtype;
    a.qsb = q_strides->sb;
    a.qsh = q_strides->sh;
    a.qst = q_strides->st;
    a.B = shape->B;
    a.Hq = shape->Hq;
    a.W = shape->W;
    a.d = shape->d;
    a.n = n;
    a.scale = query_scale(shape->d);
    a.rows = rows;
    a.q_last = q_last;
    return status_of(launch_window_rows(a, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_shape_scores(const mmskv_shape* shape, int32_t kind, int32_t window, int32_t pool, int32_t sinks,
                           const float* mass, float* score, void* stream) {
    if (shape == nullptr) return MMSKV_EINVAL;
    if (shape->B < 1 || shape->B > 65535 || shape->Hkv < 1 || shape->Hkv > 65535 || shape->T < 1)
        return MMSKV_EINVAL;
    if (score == nullptr || !aligned(score, 4)) return MMSKV_EINVAL;
    if (kind < MMSKV_SHAPE_SNAPKV || kind > MMSKV_SHAPE_SINKS) return MMSKV_EINVAL;
    if (kind != MMSKV_SHAPE_STREAMING && (mass == nullptr || !aligned(mass, 4))) return MMSKV_EINVAL;
    if (window < 0 || window > shape->T || sinks < 0 || pool < 1 || pool % 2 == 0) return MMSKV_EINVAL;
    if (shape->T > (1 << 24)) return MMSKV_EUNSUPPORTED;
    ShapeArgs a;
    a.mass = mass;
    a.score = score;
    a.B = shape->B;
    a.Hkv = shape->Hkv;
    a.T = shape->T;
    a.kind = kind;
    a.window = window;
    a.pool = pool;
    a.sinks = sinks;
    return status_of(launch_shape_scores(a, static_cast<hipStream_t>(stream)));
}

size_t mmshiftkv_hidden_stats_workspace(const mmskv_hshape* shape) {
    if (check_hshape(shape)) return 0;
    return hidden_stats_ws(shape);
}

int mmshiftkv_hidden_stats(const mmskv_hshape* shape, int32_t std_ddof, const void* hidden, int32_t dtype,
                           int64_t sb, int64_t st, double* stats, void* workspace, size_t workspace_bytes,
                           void* stream) {
    int rc = check_hshape(shape);
    if (rc) return rc;
    const int eb = elem_bytes(dtype);
    if (eb == 0 || hidden == nullptr || stats == nullptr) return MMSKV_EINVAL;
    if (std_ddof != 0 && std_ddof != 1) return MMSKV_EINVAL;
    if (shape->T - std_ddof < 1) return MMSKV_EINVAL;
    if (sb < 0 || st < 0 || !aligned(hidden, 16) || (sb * eb) % 16 || (st * eb) % 16) return MMSKV_EINVAL;
    if (!aligned(stats, 8)) return MMSKV_EINVAL;
    if (workspace == nullptr || !aligned(workspace, kAlign) || workspace_bytes < hidden_stats_ws(shape))
        return MMSKV_EWORKSPACE;
    HiddenArgs a = {};
    a.hidden = hidden;
    a.dtype = dtype;
    a.sb = sb;
    a.st = st;
    a.B = shape->B;
    a.T = shape->T;
    a.D = shape->D;
    a.chunk = kHiddenChunk;
    a.n_chunks = (shape->T + kHiddenChunk - 1) / kHiddenChunk;
    a.ddof = std_ddof;
    a.partial = static_cast<double2*>(workspace);
    a.stats = stats;
    return status_of(launch_hidden_stats(a, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_hidden_proxies(const mmskv_hshape* shape, const mmskv_params* params, const double* stats,
                             uint16_t* hp, void* stream) {
    int rc = check_hshape(shape);
    if (rc) return rc;
    if (params == nullptr || stats == nullptr || hp == nullptr) return MMSKV_EINVAL;
    if (params->P < 1 || !(params->gamma >= 0.0) || !isfinite(params->gamma)) return MMSKV_EINVAL;
    if (params->layer < 0 || params->layer > 65535) return MMSKV_EINVAL;
    if (!aligned(stats, 8) || !aligned(hp, 8)) return MMSKV_EINVAL;
    HiddenArgs a = {};
    a.B = shape->B;
    a.T = shape->T;
    a.D = shape->D;
    a.stats = const_cast<double*>(stats);
    a.hp = hp;
    a.P = params->P;
    a.layer = params->layer;
    a.gamma = params->gamma;
    a.key0 = static_cast<uint32_t>(params->seed & 0xFFFFFFFFull);
    a.key1 = static_cast<uint32_t>(params->seed >> 32);
    return status_of(launch_hidden_proxies(a, static_cast<hipStream_t>(stream)));
}

int mmshiftkv_project_proxies(const mmskv_hshape* shape, int32_t P, int32_t Hq, int32_t d, const uint16_t* hp,
                              const uint16_t* wq, const float* rope_cos, const float* rope_sin,
                              uint16_t* proxies, void* stream) {
    int rc = check_hshape(shape);
    if (rc) return rc;
    if (P < 1 || Hq < 1 || hp == nullptr || wq == nullptr || proxies == nullptr) return MMSKV_EINVAL;
    if (d != 64 && d != 128) return MMSKV_EUNSUPPORTED;
    if ((rope_cos == nullptr) != (rope_sin == nullptr)) return MMSKV_EINVAL;
    if (!aligned(hp, 16) || !aligned(wq, 16) || !aligned(proxies, 16)) return MMSKV_EINVAL;
    if (rope_cos && (!aligned(rope_cos, 4) || !aligned(rope_sin, 4))) return MMSKV_EINVAL;
    const int64_t M = static_cast<int64_t>(shape->B) * P, N = static_cast<int64_t>(Hq) * d;
    if (M > (1 << 30) || N > (1 << 30)) return MMSKV_EINVAL;
    ProjectArgs a = {};
    a.a = hp;
    a.w = wq;
    a.cos = rope_cos;
    a.sin = rope_sin;
    a.out = proxies;
    a.M = static_cast<int>(M);
    a.N = static_cast<int>(N);
    a.K = shape->D;
    a.P = P;
    a.Hq = Hq;
    a.d = d;
    a.scale = query_scale(d);
    return status_of(launch_project(a, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

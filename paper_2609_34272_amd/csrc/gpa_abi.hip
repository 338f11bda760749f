// C ABI of libgpa (declared in include/gpa.h): argument validation, workspace
// layout, kernel sequencing and optional per-kernel timing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "gpa.h"
#include "gpa_launch.h"

namespace gpa {

LaunchEvents& launch_events() {
    static thread_local LaunchEvents e;
    return e;
}

}  // namespace gpa

namespace {

thread_local std::string g_last_error;

gpa_status fail(gpa_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

struct Buf {
    const void* p;
    size_t bytes;
    const char* name;
};

bool overlap(const Buf& a, const Buf& b) {
    const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes;
    const uintptr_t b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
    return a.bytes && b.bytes && a0 < b1 && b0 < a1;
}

constexpr size_t kAlign = 256;
size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

gpa_status check_shape(int64_t B, int64_t H, int64_t N, int64_t d, float scale) {
    if (B < 1 || H < 1 || N < 1)
        return fail(GPA_EINVAL, "B, H, N must be >= 1 (got %lld, %lld, %lld)", (long long)B,
                    (long long)H, (long long)N);
    if (d != 64 && d != 128)
        return fail(GPA_ENOTSUP, "head dimension %lld not supported (64 or 128)", (long long)d);
    const double elems = (double)B * (double)H * (double)N * (double)d;
    if (elems >= 2147483648.0)
        return fail(GPA_EINVAL, "B*H*N*d = %.0f exceeds 2^31 - 1", elems);
    if (!std::isfinite(scale) || !(scale > 0.f))
        return fail(GPA_EINVAL, "scale must be finite and > 0 (got %g)", (double)scale);
    return GPA_OK;
}

gpa_status check_ptrs(const std::vector<Buf>& ins, const std::vector<Buf>& outs) {
    for (const auto* list : {&ins, &outs})
        for (const Buf& b : *list) {
            if (!b.p) return fail(GPA_EINVAL, "%s is NULL", b.name);
            if ((uintptr_t)b.p % 16) return fail(GPA_EINVAL, "%s is not 16-byte aligned", b.name);
        }
    for (size_t i = 0; i < outs.size(); ++i) {
        for (const Buf& b : ins)
            if (overlap(outs[i], b))
                return fail(GPA_EINVAL, "%s overlaps %s", outs[i].name, b.name);
        for (size_t j = i + 1; j < outs.size(); ++j)
            if (overlap(outs[i], outs[j]))
                return fail(GPA_EINVAL, "%s overlaps %s", outs[i].name, outs[j].name);
    }
    return GPA_OK;
}

// ---------------------------------------------------------------- timing
struct ProfRec {
    int id;
    hipEvent_t a, b;
};
bool g_prof = false;
std::vector<ProfRec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// With timing on, the launcher's kernel records the pair of events at its own
// start and end (launch_kernel), so each record is one kernel's duration.
template <class F>
hipError_t timed(int id, F&& launch) {
    if (!g_prof) return launch();
    hipEvent_t a = take_event(), b = take_event();
    gpa::launch_events() = {a, b};
    const hipError_t e = launch();
    gpa::launch_events() = {};
    if (a && b) g_recs.push_back({id, a, b});
    return e;
}

gpa_status launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(GPA_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
    return GPA_OK;
}

// Workspace of the atomic schedule: the per-tile statistics block (as in
// bwd_layout_rows), the FP32 [B,H,N,d] accumulator A; in the GProj modes the
// FP32 accumulator B and the FP32 [B,H,N] row masses rho, m; in gproj mode
// the FP32 [B,H,N,d] dK^acc and the BF16 -z shaped like Q.
struct AtomicLayout {
    size_t ts, a, b, rho, m, dkacc, z, total;
};

AtomicLayout atomic_layout(int64_t B, int64_t H, int64_t N, int64_t d, int mode) {
    const size_t T = (size_t)(N + 63) / 64;
    const size_t rows = (size_t)B * H * N;
    const size_t big = round_up(rows * (size_t)d * sizeof(float));
    const size_t row = round_up(rows * sizeof(float));
    AtomicLayout l{};
    size_t o = 0;
    l.ts = o;
    o += round_up((size_t)B * H * T * 128 * sizeof(float));
    l.a = o;
    o += big;
    if (mode >= 1) {
        l.b = o;
        o += big;
        l.rho = o;
        o += row;
        l.m = o;
        o += row;
    }
    if (mode == 2) {
        l.dkacc = o;
        o += big;
        l.z = o;
        o += round_up(rows * (size_t)d * 2);
    }
    l.total = o;
    return l;
}

struct BwdLayout {
    size_t D, rho, m, lam, ts, z, dkp, dvp, total;
};

// Four FP32 row statistics over the query-head rows ([B,Hq,N]; packed
// sequences [Hq,total]); per problem (query head of one sequence) and 64-row
// query tile a 512-byte block of log2-scaled LSE and D (FP32 [problems, T, 2,
// 64], T = the longest sequence rounded up to 64, over 64) that the key-major
// pass stages with the tile; then (gproj mode only) the BF16 tensor
// -z = BF16(-lambda q), shaped like Q, that the key correction contracts; then,
// for grouped-query attention (Hq > Hkv) only, the FP32 per-query-head
// contributions to dK and dV (Hq heads over the key rows) that the group sum
// adds.
BwdLayout bwd_layout_rows(size_t qrows, size_t krows, size_t problems, int64_t Nmax, int64_t d,
                          int mode, bool grouped) {
    const size_t row = round_up(qrows * sizeof(float));
    const size_t T = (size_t)(Nmax + 63) / 64;
    const size_t tstats = round_up(problems * T * 128 * sizeof(float));
    const size_t part = grouped ? round_up(krows * (size_t)d * sizeof(float)) : 0;
    BwdLayout L;
    L.D = 0;
    L.rho = row;
    L.m = 2 * row;
    L.lam = 3 * row;
    L.ts = 4 * row;
    L.z = L.ts + tstats;
    L.dkp = L.z + (mode == 2 ? round_up(qrows * (size_t)d * 2) : 0);
    L.dvp = L.dkp + part;
    L.total = L.dvp + part;
    return L;
}

BwdLayout bwd_layout(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d, int mode) {
    const size_t rows = (size_t)B * Hq * N;
    return bwd_layout_rows(rows, rows, (size_t)B * Hq, N, d, mode, Hq > Hkv);
}

// Enqueue the backward passes once the arguments are validated: the
// query-major pass, the key-major pass and, for grouped-query attention, the
// group sum of the per-query-head dK, dV contributions.  krows is the number
// of query-head rows over the keys (Hq x key rows: the extent of the
// group-sum partials).
gpa_status run_bwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const uint16_t* O,
                   const float* LSE, const uint16_t* dO, uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                   const gpa::Shape& sh, const BwdLayout& L, size_t krows, int mode,
                   void* workspace, hipStream_t st) {
    char* ws = (char*)workspace;
    float* Drow = (float*)(ws + L.D);
    float* rho = (float*)(ws + L.rho);
    float* msum = (float*)(ws + L.m);
    float* lam = (float*)(ws + L.lam);
    float* tstats = (float*)(ws + L.ts);
    uint16_t* zbuf = mode == 2 ? (uint16_t*)(ws + L.z) : nullptr;
    float* dkp = sh.G > 1 ? (float*)(ws + L.dkp) : nullptr;
    float* dvp = sh.G > 1 ? (float*)(ws + L.dvp) : nullptr;

    gpa_status s = launched(timed(gpa::kKBwdDq,
                                  [&] {
                                      return gpa::launch_bwd_dq(Q, K, V, O, dO, LSE, Drow, tstats,
                                                                dQ, rho, msum, lam, zbuf, mode, sh,
                                                                st);
                                  }),
                            "bwd_dq");
    if (s != GPA_OK) return s;
    s = launched(timed(gpa::kKBwdDkdv,
                       [&] {
                           return gpa::launch_bwd_dkdv(Q, K, V, dO, tstats, zbuf, dK, dV, dkp, dvp,
                                                       mode, sh, st);
                       }),
                 "bwd_dkdv");
    if (s != GPA_OK || sh.G == 1) return s;
    // The group sum sees the partials as G consecutive query heads of
    // krows / Hq key rows each per key/value head.
    gpa::Shape gs = sh;
    gs.BH = sh.cu ? sh.Hq : sh.BH;
    gs.N = (int)(krows / (size_t)gs.BH);
    return launched(timed(gpa::kKGroupSum,
                          [&] { return gpa::launch_bwd_group_sum(dkp, dvp, dK, dV, gs, st); }),
                    "group_sum");
}

gpa_status check_heads(int64_t Hq, int64_t Hkv) {
    if (Hkv < 1 || Hq < 1 || Hq % Hkv != 0)
        return fail(GPA_EINVAL, "query heads %lld must be a positive multiple of key/value heads %lld",
                    (long long)Hq, (long long)Hkv);
    return GPA_OK;
}

// Packed variable-length sequences: the query side and the key side each
// have offsets, a total and a longest run.  Key offsets NULL means the query
// offsets, which asks for the same total and longest run.
struct Varlen {
    const int32_t* cu_q;
    const int32_t* cu_k;
    int64_t nseq, total_q, total_k, Hq, Hkv, max_q, max_k, d;
};

gpa_status check_varlen(const Varlen& v, float scale) {
    if (v.nseq < 1 || v.total_q < 1 || v.max_q < 1 || v.max_q > v.total_q)
        return fail(GPA_EINVAL,
                    "need nseq >= 1, total_q >= 1 and 1 <= max_seqlen_q <= total_q "
                    "(got %lld, %lld, %lld)",
                    (long long)v.nseq, (long long)v.total_q, (long long)v.max_q);
    if (v.total_k < 1 || v.max_k < 1 || v.max_k > v.total_k)
        return fail(GPA_EINVAL, "need total_k >= 1 and 1 <= max_seqlen_k <= total_k (got %lld, %lld)",
                    (long long)v.total_k, (long long)v.max_k);
    if (v.cu_k == v.cu_q && (v.total_k != v.total_q || v.max_k != v.max_q))
        return fail(GPA_EINVAL, "shared offsets need total_k == total_q and max_seqlen_k == max_seqlen_q");
    gpa_status s = check_shape(1, v.Hq, v.total_q, v.d, scale);
    if (s != GPA_OK) return s;
    if ((s = check_shape(1, v.Hq, v.total_k, v.d, scale)) != GPA_OK) return s;
    if ((s = check_heads(v.Hq, v.Hkv)) != GPA_OK) return s;
    if (!v.cu_q) return fail(GPA_EINVAL, "cu_seqlens_q is NULL");
    if ((uintptr_t)v.cu_q % 4 || (uintptr_t)v.cu_k % 4)
        return fail(GPA_EINVAL, "sequence offsets are not 4-byte aligned");
    const int64_t longest = v.max_q > v.max_k ? v.max_q : v.max_k;
    const double grid = (double)v.nseq * (double)v.Hq * (double)((longest + 63) / 64);
    if (grid >= 2147483648.0 || (double)v.nseq * v.Hq >= 2147483648.0)
        return fail(GPA_EINVAL, "nseq * Hq * ceil(max_seqlen / 64) = %.0f exceeds 2^31 - 1", grid);
    return GPA_OK;
}

// The sequence offsets are an input: no output may overlap them.
gpa_status check_cu_overlap(const Varlen& v, const std::vector<Buf>& outs) {
    const Buf c[2] = {{v.cu_q, 4 * (size_t)(v.nseq + 1), "cu_seqlens_q"},
                      {v.cu_k, 4 * (size_t)(v.nseq + 1), "cu_seqlens_k"}};
    for (const Buf& b : outs)
        for (const Buf& cb : c)
            if (overlap(b, cb)) return fail(GPA_EINVAL, "%s overlaps %s", b.name, cb.name);
    return GPA_OK;
}

gpa::Shape varlen_shape(const Varlen& v, int causal, float scale) {
    gpa::Shape sh{(int)(v.nseq * v.Hq), (int)v.max_q, (int)v.d, causal ? 1 : 0, scale,
                  (int)(v.Hq / v.Hkv)};
    sh.cu = v.cu_q;
    sh.Hq = (int)v.Hq;
    sh.total = (int)v.total_q;
    sh.cu_k = v.cu_k;
    sh.total_k = (int)v.total_k;
    sh.Nk = (int)v.max_k;
    return sh;
}

// ------------------------------------------------- no-allocation scratch
// Device memory of gpa_attn_bwd_noalloc: the backward's workspace (row
// statistics, per-tile statistics, z) for callers that cannot allocate.  One
// copy per GPU, held until the process ends; every call on a GPU shares it.
constexpr size_t kScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

// Host code never passes `scratch` itself to a kernel: on the host the name
// is a stand-in, not a device address.  Its address on each device comes
// from hipGetSymbolAddress, taken once per device with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

gpa_status scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(GPA_EHIP, "hipGetDevice failed: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(GPA_EHIP, "device %d beyond the %d devices the scratch table covers", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(GPA_EHIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return GPA_OK;
}

BwdLayout varlen_layout(const Varlen& v, int mode) {
    return bwd_layout_rows((size_t)v.Hq * v.total_q, (size_t)v.Hq * v.total_k,
                           (size_t)v.nseq * v.Hq, v.max_q, v.d, mode, v.Hq > v.Hkv);
}
// Fused FP32 baseline workspace: the saved FP32 output O32 [B,H,N,d], the
// scaled row maximum and the inverse normaliser [B,H,N] each, and the
// per-tile statistics the key-major pass stages ([B*H, T, 3, 64]).
struct F32Layout {
    size_t o32, mrow, linv, ts, total;
};
F32Layout f32_layout(int64_t B, int64_t H, int64_t N, int64_t d) {
    const size_t rows = (size_t)B * H * N;
    const size_t T = (size_t)(N + 63) / 64;
    F32Layout L;
    L.o32 = 0;
    L.mrow = round_up(rows * d * 4);
    L.linv = L.mrow + round_up(rows * 4);
    L.ts = L.linv + round_up(rows * 4);
    L.total = L.ts + round_up((size_t)B * H * T * 192 * 4);
    return L;
}

}  // namespace

extern "C" {

const char* gpa_version(void) { return "gpa 0.1.0 gfx950"; }

const char* gpa_status_str(gpa_status s) {
    switch (s) {
        case GPA_OK: return "GPA_OK";
        case GPA_EINVAL: return "GPA_EINVAL: invalid argument";
        case GPA_ENOTSUP: return "GPA_ENOTSUP: unsupported head dimension";
        case GPA_EWORKSPACE: return "GPA_EWORKSPACE: workspace missing or too small";
        case GPA_EHIP: return "GPA_EHIP: HIP launch failure";
    }
    return "unknown gpa_status";
}

const char* gpa_last_error(void) { return g_last_error.c_str(); }

gpa_status gpa_attn_fwd_gqa(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            uint16_t* O, float* LSE, int64_t B, int64_t Hq, int64_t Hkv,
                            int64_t N, int64_t d, int causal, float scale, void* stream) {
    gpa_status s = check_shape(B, Hq, N, d, scale);
    if (s != GPA_OK) return s;
    if ((s = check_heads(Hq, Hkv)) != GPA_OK) return s;
    const size_t tq = (size_t)B * Hq * N * d * 2, tkv = (size_t)B * Hkv * N * d * 2;
    const size_t lb = (size_t)B * Hq * N * 4;
    s = check_ptrs({{Q, tq, "Q"}, {K, tkv, "K"}, {V, tkv, "V"}}, {{O, tq, "O"}, {LSE, lb, "LSE"}});
    if (s != GPA_OK) return s;
    const gpa::Shape sh{(int)(B * Hq), (int)N, (int)d, causal ? 1 : 0, scale, (int)(Hq / Hkv)};
    hipStream_t st = (hipStream_t)stream;
    return launched(timed(gpa::kKFwd, [&] { return gpa::launch_fwd(Q, K, V, O, LSE, sh, st); }),
                    "fwd_sbs");
}

gpa_status gpa_attn_fwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V, uint16_t* O,
                        float* LSE, int64_t B, int64_t H, int64_t N, int64_t d, int causal,
                        float scale, void* stream) {
    return gpa_attn_fwd_gqa(Q, K, V, O, LSE, B, H, H, N, d, causal, scale, stream);
}

gpa_status gpa_attn_fwd_fma(const uint16_t* Q, const uint16_t* K, const uint16_t* V, uint16_t* O,
                            float* LSE, int64_t B, int64_t H, int64_t N, int64_t d, int causal,
                            float scale, void* stream) {
    gpa_status s = check_shape(B, H, N, d, scale);
    if (s != GPA_OK) return s;
    const size_t tb = (size_t)B * H * N * d * 2, lb = (size_t)B * H * N * 4;
    s = check_ptrs({{Q, tb, "Q"}, {K, tb, "K"}, {V, tb, "V"}}, {{O, tb, "O"}, {LSE, lb, "LSE"}});
    if (s != GPA_OK) return s;
    const gpa::Shape sh{(int)(B * H), (int)N, (int)d, causal ? 1 : 0, scale, 1};
    hipStream_t st = (hipStream_t)stream;
    return launched(
        timed(gpa::kKFwd, [&] { return gpa::launch_fwd(Q, K, V, O, LSE, sh, st, true); }),
        "fwd_fma");
}

size_t gpa_attn_bwd_gqa_workspace_bytes(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t d,
                                        int mode) {
    if (mode < 0 || mode > 2) return 0;
    if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || N < 1 || (d != 64 && d != 128)) return 0;
    if ((double)B * Hq * N * d >= 2147483648.0) return 0;
    return bwd_layout(B, Hq, Hkv, N, d, mode).total;
}

size_t gpa_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d, int mode) {
    return gpa_attn_bwd_gqa_workspace_bytes(B, H, H, N, d, mode);
}

gpa_status gpa_bwd_stats_offsets(int64_t B, int64_t H, int64_t N, int64_t d, int mode,
                                 size_t* off_D, size_t* off_rho, size_t* off_m,
                                 size_t* off_lambda) {
    if (gpa_attn_bwd_workspace_bytes(B, H, N, d, mode) == 0)
        return fail(GPA_EINVAL, "invalid shape or mode");
    const BwdLayout L = bwd_layout(B, H, H, N, d, mode);
    if (off_D) *off_D = L.D;
    if (off_rho) *off_rho = L.rho;
    if (off_m) *off_m = L.m;
    if (off_lambda) *off_lambda = L.lam;
    return GPA_OK;
}

gpa_status gpa_attn_bwd_gqa(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                            const uint16_t* O, const float* LSE, const uint16_t* dO,
                            uint16_t* dQ, uint16_t* dK, uint16_t* dV, int64_t B, int64_t Hq,
                            int64_t Hkv, int64_t N, int64_t d, int causal, float scale, int mode,
                            void* workspace, size_t workspace_bytes, void* stream) {
    gpa_status s = check_shape(B, Hq, N, d, scale);
    if (s != GPA_OK) return s;
    if ((s = check_heads(Hq, Hkv)) != GPA_OK) return s;
    if (mode < 0 || mode > 2) return fail(GPA_EINVAL, "mode %d is not 0, 1 or 2", mode);
    const size_t need = gpa_attn_bwd_gqa_workspace_bytes(B, Hq, Hkv, N, d, mode);
    if (!workspace || workspace_bytes < need)
        return fail(GPA_EWORKSPACE, "workspace %p of %zu bytes; %zu needed", workspace,
                    workspace_bytes, need);
    if ((uintptr_t)workspace % kAlign)
        return fail(GPA_EWORKSPACE, "workspace is not %zu-byte aligned", kAlign);
    const size_t tq = (size_t)B * Hq * N * d * 2, tkv = (size_t)B * Hkv * N * d * 2;
    const size_t lb = (size_t)B * Hq * N * 4;
    s = check_ptrs({{Q, tq, "Q"}, {K, tkv, "K"}, {V, tkv, "V"}, {O, tq, "O"}, {LSE, lb, "LSE"},
                    {dO, tq, "dO"}},
                   {{dQ, tq, "dQ"}, {dK, tkv, "dK"}, {dV, tkv, "dV"}, {workspace, need, "workspace"}});
    if (s != GPA_OK) return s;

    const gpa::Shape sh{(int)(B * Hq), (int)N, (int)d, causal ? 1 : 0, scale, (int)(Hq / Hkv)};
    return run_bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, sh, bwd_layout(B, Hq, Hkv, N, d, mode),
                   (size_t)B * Hq * N, mode, workspace, (hipStream_t)stream);
}

gpa_status gpa_attn_bwd(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* O, const float* LSE, const uint16_t* dO, uint16_t* dQ,
                        uint16_t* dK, uint16_t* dV, int64_t B, int64_t H, int64_t N, int64_t d,
                        int causal, float scale, int mode, void* workspace,
                        size_t workspace_bytes, void* stream) {
    return gpa_attn_bwd_gqa(Q, K, V, O, LSE, dO, dQ, dK, dV, B, H, H, N, d, causal, scale, mode,
                            workspace, workspace_bytes, stream);
}


size_t gpa_attn_bwd_noalloc_max_bytes(void) { return kScratchBytes; }

gpa_status gpa_attn_bwd_noalloc(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                                const uint16_t* O, const float* LSE, const uint16_t* dO,
                                uint16_t* dQ, uint16_t* dK, uint16_t* dV, int64_t B, int64_t H,
                                int64_t N, int64_t d, int causal, float scale, int mode,
                                void* stream) {
    gpa_status s = check_shape(B, H, N, d, scale);
    if (s != GPA_OK) return s;
    if (mode < 0 || mode > 2) return fail(GPA_EINVAL, "mode %d is not 0, 1 or 2", mode);
    const size_t need = gpa_attn_bwd_workspace_bytes(B, H, N, d, mode);
    if (need > kScratchBytes)
        return fail(GPA_EWORKSPACE,
                    "this shape needs %zu bytes of scratch; gpa_attn_bwd_noalloc holds at most %zu "
                    "(use gpa_attn_bwd with a workspace)",
                    need, kScratchBytes);
    const size_t tb = (size_t)B * H * N * d * 2, lb = (size_t)B * H * N * 4;
    s = check_ptrs({{Q, tb, "Q"}, {K, tb, "K"}, {V, tb, "V"}, {O, tb, "O"}, {LSE, lb, "LSE"},
                    {dO, tb, "dO"}},
                   {{dQ, tb, "dQ"}, {dK, tb, "dK"}, {dV, tb, "dV"}});
    if (s != GPA_OK) return s;
    void* ws = nullptr;
    if ((s = scratch_address(&ws)) != GPA_OK) return s;
    const gpa::Shape sh{(int)(B * H), (int)N, (int)d, causal ? 1 : 0, scale, 1};
    return run_bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, sh, bwd_layout(B, H, H, N, d, mode),
                   (size_t)B * H * N, mode, ws, (hipStream_t)stream);
}

size_t gpa_attn_bwd_atomic_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d,
                                           int mode) {
    if (B < 1 || H < 1 || N < 1 || (d != 64 && d != 128) || mode < 0 || mode > 2) return 0;
    if ((double)B * H * N * d >= 2147483648.0) return 0;
    const AtomicLayout l = atomic_layout(B, H, N, d, mode);
    return l.total;
}

gpa_status gpa_attn_bwd_atomic(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               const uint16_t* O, const float* LSE, const uint16_t* dO,
                               uint16_t* dQ, uint16_t* dK, uint16_t* dV, int64_t B, int64_t H,
                               int64_t N, int64_t d, int causal, float scale, int mode,
                               void* workspace, size_t workspace_bytes, void* stream) {
    gpa_status s = check_shape(B, H, N, d, scale);
    if (s != GPA_OK) return s;
    if (mode < 0 || mode > 2) return fail(GPA_EINVAL, "mode %d is not 0, 1 or 2", mode);
    const size_t need = gpa_attn_bwd_atomic_workspace_bytes(B, H, N, d, mode);
    if (!workspace || workspace_bytes < need)
        return fail(GPA_EWORKSPACE, "workspace %p of %zu bytes; %zu needed", workspace,
                    workspace_bytes, need);
    if ((uintptr_t)workspace % kAlign)
        return fail(GPA_EWORKSPACE, "workspace is not %zu-byte aligned", kAlign);
    const size_t tb = (size_t)B * H * N * d * 2, lb = (size_t)B * H * N * 4;
    s = check_ptrs({{Q, tb, "Q"}, {K, tb, "K"}, {V, tb, "V"}, {O, tb, "O"}, {LSE, lb, "LSE"},
                    {dO, tb, "dO"}},
                   {{dQ, tb, "dQ"}, {dK, tb, "dK"}, {dV, tb, "dV"}, {workspace, need, "workspace"}});
    if (s != GPA_OK) return s;
    const gpa::Shape sh{(int)(B * H), (int)N, (int)d, causal ? 1 : 0, scale, 1};
    hipStream_t st = (hipStream_t)stream;
    const AtomicLayout l = atomic_layout(B, H, N, d, mode);
    char* w = (char*)workspace;
    float* TS = (float*)(w + l.ts);
    gpa::AtomicAcc acc;
    acc.A = (float*)(w + l.a);
    if (mode >= 1) {
        acc.B = (float*)(w + l.b);
        acc.rho = (float*)(w + l.rho);
        acc.m = (float*)(w + l.m);
    }
    if (mode == 2) acc.dKacc = (float*)(w + l.dkacc);
    uint16_t* Zneg = mode == 2 ? (uint16_t*)(w + l.z) : nullptr;
    s = launched(timed(gpa::kKBwdPre,
                       [&] { return gpa::launch_bwd_pre(O, dO, LSE, TS, acc, sh, st); }),
                 "bwd_pre");
    if (s != GPA_OK) return s;
    s = launched(timed(gpa::kKBwdFused,
                       [&] {
                           return gpa::launch_bwd_fused(Q, K, V, dO, TS, dK, dV, acc, mode, sh,
                                                        st);
                       }),
                 "bwd_fused");
    if (s != GPA_OK) return s;
    if (mode == 0)
        return launched(timed(gpa::kKBwdFinal,
                              [&] { return gpa::launch_bwd_dq_finalize(acc.A, dQ, sh, st); }),
                        "bwd_dq_finalize");
    s = launched(timed(gpa::kKBwdFinal,
                       [&] {
                           return gpa::launch_bwd_gproj_finalize(acc, Q, dQ, Zneg, nullptr, sh,
                                                                 st);
                       }),
                 "bwd_gproj_finalize");
    if (s != GPA_OK || mode == 1) return s;
    return launched(timed(gpa::kKBwdCorr,
                          [&] {
                              return gpa::launch_bwd_dk_corr(Q, K, TS, Zneg, acc.dKacc, dK, sh, st);
                          }),
                    "bwd_dk_corr");
}

gpa_status gpa_attn_fwd_varlen(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               uint16_t* O, float* LSE, const int32_t* cu_seqlens_q,
                               const int32_t* cu_seqlens_k, int64_t nseq, int64_t total_q,
                               int64_t total_k, int64_t Hq, int64_t Hkv, int64_t max_seqlen_q,
                               int64_t max_seqlen_k, int64_t d, int causal, float scale,
                               void* stream) {
    const Varlen v{cu_seqlens_q, cu_seqlens_k ? cu_seqlens_k : cu_seqlens_q, nseq, total_q,
                   total_k, Hq, Hkv, max_seqlen_q, max_seqlen_k, d};
    gpa_status s = check_varlen(v, scale);
    if (s != GPA_OK) return s;
    const size_t tq = (size_t)Hq * total_q * d * 2, tkv = (size_t)Hkv * total_k * d * 2;
    const size_t lb = (size_t)Hq * total_q * 4;
    const std::vector<Buf> outs = {{O, tq, "O"}, {LSE, lb, "LSE"}};
    s = check_ptrs({{Q, tq, "Q"}, {K, tkv, "K"}, {V, tkv, "V"}}, outs);
    if (s != GPA_OK) return s;
    if ((s = check_cu_overlap(v, outs)) != GPA_OK) return s;
    const gpa::Shape sh = varlen_shape(v, causal, scale);
    hipStream_t st = (hipStream_t)stream;
    return launched(timed(gpa::kKFwd, [&] { return gpa::launch_fwd(Q, K, V, O, LSE, sh, st); }),
                    "fwd_sbs");
}

size_t gpa_attn_bwd_varlen_workspace_bytes(int64_t nseq, int64_t total_q, int64_t total_k,
                                           int64_t Hq, int64_t Hkv, int64_t max_seqlen_q,
                                           int64_t max_seqlen_k, int64_t d, int mode) {
    if (mode < 0 || mode > 2) return 0;
    if (nseq < 1 || total_q < 1 || max_seqlen_q < 1 || max_seqlen_q > total_q) return 0;
    if (total_k < 1 || max_seqlen_k < 1 || max_seqlen_k > total_k) return 0;
    if (Hq < 1 || Hkv < 1 || Hq % Hkv || (d != 64 && d != 128)) return 0;
    if ((double)Hq * total_q * d >= 2147483648.0 || (double)Hq * total_k * d >= 2147483648.0)
        return 0;
    const int64_t longest = max_seqlen_q > max_seqlen_k ? max_seqlen_q : max_seqlen_k;
    if ((double)nseq * Hq * (double)((longest + 63) / 64) >= 2147483648.0) return 0;
    const Varlen v{nullptr, nullptr, nseq, total_q, total_k, Hq, Hkv, max_seqlen_q, max_seqlen_k, d};
    return varlen_layout(v, mode).total;
}

gpa_status gpa_attn_bwd_varlen(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                               const uint16_t* O, const float* LSE, const uint16_t* dO,
                               uint16_t* dQ, uint16_t* dK, uint16_t* dV,
                               const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                               int64_t nseq, int64_t total_q, int64_t total_k, int64_t Hq,
                               int64_t Hkv, int64_t max_seqlen_q, int64_t max_seqlen_k, int64_t d,
                               int causal, float scale, int mode, void* workspace,
                               size_t workspace_bytes, void* stream) {
    const Varlen v{cu_seqlens_q, cu_seqlens_k ? cu_seqlens_k : cu_seqlens_q, nseq, total_q,
                   total_k, Hq, Hkv, max_seqlen_q, max_seqlen_k, d};
    gpa_status s = check_varlen(v, scale);
    if (s != GPA_OK) return s;
    if (mode < 0 || mode > 2) return fail(GPA_EINVAL, "mode %d is not 0, 1 or 2", mode);
    const size_t need = gpa_attn_bwd_varlen_workspace_bytes(nseq, total_q, total_k, Hq, Hkv,
                                                            max_seqlen_q, max_seqlen_k, d, mode);
    if (!workspace || workspace_bytes < need)
        return fail(GPA_EWORKSPACE, "workspace %p of %zu bytes; %zu needed", workspace,
                    workspace_bytes, need);
    if ((uintptr_t)workspace % kAlign)
        return fail(GPA_EWORKSPACE, "workspace is not %zu-byte aligned", kAlign);
    const size_t tq = (size_t)Hq * total_q * d * 2, tkv = (size_t)Hkv * total_k * d * 2;
    const size_t lb = (size_t)Hq * total_q * 4;
    const std::vector<Buf> outs = {
        {dQ, tq, "dQ"}, {dK, tkv, "dK"}, {dV, tkv, "dV"}, {workspace, need, "workspace"}};
    s = check_ptrs({{Q, tq, "Q"}, {K, tkv, "K"}, {V, tkv, "V"}, {O, tq, "O"}, {LSE, lb, "LSE"},
                    {dO, tq, "dO"}},
                   outs);
    if (s != GPA_OK) return s;
    if ((s = check_cu_overlap(v, outs)) != GPA_OK) return s;
    const gpa::Shape sh = varlen_shape(v, causal, scale);
    return run_bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, sh, varlen_layout(v, mode),
                   (size_t)Hq * total_k, mode, workspace, (hipStream_t)stream);
}

size_t gpa_fp32_attn_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d) {
    if (B < 1 || H < 1 || N < 1 || (d != 64 && d != 128)) return 0;
    if ((double)B * H * N * d >= 2147483648.0) return 0;
    return f32_layout(B, H, N, d).total;
}

gpa_status gpa_fp32_attn(const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         const uint16_t* dO, uint16_t* O, float* LSE, uint16_t* dQ, uint16_t* dK,
                         uint16_t* dV, int64_t B, int64_t H, int64_t N, int64_t d, int causal,
                         float scale, void* workspace, size_t workspace_bytes, void* stream) {
    gpa_status s = check_shape(B, H, N, d, scale);
    if (s != GPA_OK) return s;
    const size_t need = gpa_fp32_attn_workspace_bytes(B, H, N, d);
    if (!workspace || workspace_bytes < need)
        return fail(GPA_EWORKSPACE, "workspace %p of %zu bytes; %zu needed", workspace,
                    workspace_bytes, need);
    if ((uintptr_t)workspace % kAlign)
        return fail(GPA_EWORKSPACE, "workspace is not %zu-byte aligned", kAlign);
    const size_t tb = (size_t)B * H * N * d * 2, lb = (size_t)B * H * N * 4;
    s = check_ptrs({{Q, tb, "Q"}, {K, tb, "K"}, {V, tb, "V"}, {dO, tb, "dO"}},
                   {{O, tb, "O"}, {LSE, lb, "LSE"}, {dQ, tb, "dQ"}, {dK, tb, "dK"},
                    {dV, tb, "dV"}, {workspace, need, "workspace"}});
    if (s != GPA_OK) return s;
    const gpa::Shape sh{(int)(B * H), (int)N, (int)d, causal ? 1 : 0, scale, 1};
    hipStream_t st = (hipStream_t)stream;
    const F32Layout L = f32_layout(B, H, N, d);
    char* ws = (char*)workspace;
    float* O32 = (float*)(ws + L.o32);
    float* Mrow = (float*)(ws + L.mrow);
    float* Linv = (float*)(ws + L.linv);
    float* TS = (float*)(ws + L.ts);
    s = launched(timed(gpa::kKF32Fwd,
                       [&] { return gpa::launch_f32_fwd(Q, K, V, O32, O, LSE, Mrow, Linv, sh, st); }),
                 "fp32_fwd");
    if (s != GPA_OK) return s;
    s = launched(timed(gpa::kKF32Dq,
                       [&] {
                           return gpa::launch_f32_dq(Q, K, V, dO, O32, Mrow, Linv, TS, dQ, sh, st);
                       }),
                 "fp32_dq");
    if (s != GPA_OK) return s;
    return launched(timed(gpa::kKF32Dkdv,
                          [&] { return gpa::launch_f32_dkdv(Q, K, V, dO, TS, dK, dV, sh, st); }),
                    "fp32_dkdv");
}

void gpa_profile_enable(int on) { g_prof = on != 0; }

int gpa_profile_read(double* total_ms, int64_t* launches, int n) {
    for (int i = 0; i < n; ++i) {
        if (total_ms) total_ms[i] = 0.0;
        if (launches) launches[i] = 0;
    }
    for (const ProfRec& r : g_recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess &&
            r.id < n) {
            if (total_ms) total_ms[r.id] += ms;
            if (launches) launches[r.id] += 1;
        }
        g_pool.push_back(r.a);
        g_pool.push_back(r.b);
    }
    g_recs.clear();
    return gpa::kNumKernels;
}

const char* gpa_kernel_name(int id) {
    static const char* names[gpa::kNumKernels] = {
        "fwd_sbs",   "bwd_dq",  "bwd_dkdv",        "fp32_fwd",       "fp32_dq",
        "fp32_dkdv", "group_sum", "bwd_pre", "bwd_fused", "bwd_dq_finalize", "bwd_dk_corr"};
    return (id >= 0 && id < gpa::kNumKernels) ? names[id] : "";
}

}  // extern "C"

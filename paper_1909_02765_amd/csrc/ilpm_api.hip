// C-ABI layer: argument checks, plan choice, workspace, device check and
// launch.  Declarations and contracts are in include/ilpm.h.
#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "internal.h"

// The no-alloc entry point's workspace: one fixed array per device, created
// when the code object loads and kept until the process ends (host code uses
// the address hipGetSymbolAddress returns for it, never this name).
static __device__ __align__(256) float scratch[ILPM_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace ilpm {
namespace {

constexpr int kMaxDevices = 64;
constexpr int64_t kMaxElems = 0x7fffffffLL;

std::mutex g_mu;
std::atomic<int> g_arch[kMaxDevices];  // 0 unknown, 1 gfx950, -1 other
void *g_scratch[kMaxDevices];          // device address of `scratch` per device (under g_mu)
thread_local int g_last_hip = 0;  // hipError_t behind the last ILPM_ERR_HIP of this thread

int hip_fail(hipError_t e)
{
    g_last_hip = (int)e;
    return ILPM_ERR_HIP;
}

struct Workspace {
    void *user = nullptr;
    size_t user_bytes = 0;
    void *own = nullptr;
    size_t own_bytes = 0;
    // Smaller library-owned buffers that a larger one replaced.  They are
    // never freed: a call still running, or a graph captured earlier, may use
    // them, and freeing would need a synchronisation.
    std::vector<void *> retired;
};
Workspace g_ws[kMaxDevices];

// Environment overrides, read once when the library first plans a call.
struct Overrides {
    int path = -1;          // ILPM_FORCE_PATH: -1 any, ILPM_PATH_DIRECT or ILPM_PATH_IGEMM
    int splits = 0;         // ILPM_SPLIT: input-channel splits of matrix-core plans (0 = choose)
    int tile_h = 0, tile_w = 0;  // ILPM_TILE=<h>x<w>: only variants with this output tile
};

Overrides read_overrides()
{
    Overrides o;
    if (const char *f = std::getenv("ILPM_FORCE_PATH")) {
        if (std::strcmp(f, "direct") == 0) o.path = ILPM_PATH_DIRECT;
        else if (std::strcmp(f, "igemm") == 0 || std::strcmp(f, "gemm") == 0) o.path = ILPM_PATH_IGEMM;
    }
    if (const char *e = std::getenv("ILPM_SPLIT")) o.splits = std::max(0, std::atoi(e));
    if (const char *t = std::getenv("ILPM_TILE")) {
        int h = 0, w = 0;
        if (std::sscanf(t, "%dx%d", &h, &w) == 2 && h > 0 && w > 0) {
            o.tile_h = h;
            o.tile_w = w;
        }
    }
    return o;
}

const Overrides &overrides()
{
    static const Overrides o = read_overrides();
    return o;
}

bool overlaps(const void *a, size_t an, const void *b, size_t bn)
{
    if (!a || !b || an == 0 || bn == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

// Output size along one axis, -1 when no window fits.
int64_t out_extent(int n, int k, int stride, int pad)
{
    const int64_t span = (int64_t)n + 2 * (int64_t)pad - k;
    if (span < 0) return -1;
    return span / stride + 1;
}

int check_dims(int c_in, int h, int w, int c_out, int k, int stride, int pad, ConvShape *s)
{
    if (c_in <= 0 || h <= 0 || w <= 0 || c_out <= 0 || k <= 0 || stride <= 0 || pad < 0)
        return ILPM_ERR_INVALID_ARG;
    const int64_t ho = out_extent(h, k, stride, pad);
    const int64_t wo = out_extent(w, k, stride, pad);
    if (ho < 1 || wo < 1) return ILPM_ERR_INVALID_ARG;
    if ((int64_t)c_in * h * w > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    if ((int64_t)c_out * c_in * k * k > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    if ((int64_t)c_out * ho * wo > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    if (ho > kMaxElems || wo > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    if (s) {
        s->c_in = c_in; s->h = h; s->w = w; s->c_out = c_out; s->k = k;
        s->stride = stride; s->pad = pad; s->h_out = (int)ho; s->w_out = (int)wo;
    }
    return ILPM_OK;
}

// Output bytes of a call: the conv output, or its 2x2-pooled version.
size_t out_bytes(const ConvShape &s, int epilogue)
{
    if (epilogue & ILPM_EPI_MAXPOOL2) return sizeof(float) * (size_t)s.c_out * (s.h_out / 2) * (s.w_out / 2);
    return sizeof(float) * (size_t)s.c_out * s.h_out * s.w_out;
}

int validate(const void *in, const void *w, const void *bias, const ConvShape &s, const void *out, int epilogue = 0)
{
    if (!in || !w || !out) return ILPM_ERR_INVALID_ARG;
    const size_t in_b = sizeof(float) * (size_t)s.c_in * s.h * s.w;
    const size_t w_b = sizeof(float) * (size_t)s.c_out * s.c_in * s.k * s.k;
    const size_t b_b = sizeof(float) * (size_t)s.c_out;
    const size_t o_b = out_bytes(s, epilogue);
    if (((uintptr_t)in | (uintptr_t)w | (uintptr_t)out | (uintptr_t)bias) & 3u) return ILPM_ERR_INVALID_ARG;
    if (overlaps(out, o_b, in, in_b) || overlaps(out, o_b, w, w_b) || overlaps(out, o_b, bias, b_b))
        return ILPM_ERR_INVALID_ARG;
    return ILPM_OK;
}

// The default plan: the measured best for this exact shape when a tuning
// table has it -- the table of this weight layout and epilogue first, then
// (pooled) the plain table of the same layout, then the OIHW tables -- else
// the cheapest matrix-core variant for this filter size and stride by the
// cost model, else the LDS direct kernel, else the plain one.  The
// environment overrides (read once) narrow the candidates.
int compute_plan(const ConvShape &s, ilpm_plan *p, bool prepacked, bool pooled)
{
    const Overrides &o = overrides();
    const bool any = o.path < 0 && o.splits == 0 && o.tile_h == 0;
    if (any) {
        if (pooled && prepacked && tuned_plan(s, p, true, true)) return ILPM_OK;
        if (prepacked && tuned_plan(s, p, true, false)) return ILPM_OK;
        if (pooled && tuned_plan(s, p, false, true)) return ILPM_OK;
        if (tuned_plan(s, p, false, false)) return ILPM_OK;
    }
    auto tile_ok = [&](const ilpm_plan &q) { return o.tile_h == 0 || (q.tile_h == o.tile_h && q.tile_w == o.tile_w); };
    if (o.path != ILPM_PATH_DIRECT) {
        bool found = false;
        double best = 0;
        ilpm_plan bp = {};
        for (int v = 0; v < igemm_num_variants(); ++v) {
            ilpm_plan q;
            if (!igemm_make_plan(s, v, o.splits, &q) || !tile_ok(q)) continue;
            const double c = igemm_plan_cost(s, q);
            if (!found || c < best) {
                found = true;
                best = c;
                bp = q;
            }
        }
        if (found) {
            *p = bp;
            return ILPM_OK;
        }
    }
    if (o.path == ILPM_PATH_IGEMM) return ILPM_ERR_UNSUPPORTED;
    for (int v = 0; v < direct_num_variants(); ++v) {
        ilpm_plan q;
        if (direct_make_plan(s, v, &q) && tile_ok(q)) {
            *p = q;
            return ILPM_OK;
        }
    }
    return ILPM_ERR_UNSUPPORTED;
}

// Plans already chosen, by shape: a direct-mapped table, so a call on a shape
// seen before costs one hash and one comparison instead of the table scan and
// the cost-model sweep.
struct PlanSlot {
    bool used = false;
    int mode;  // 1: prepacked weights, 2: pooled epilogue
    ConvShape s;
    int rc;
    ilpm_plan p;
};
constexpr int kPlanSlots = 512;
PlanSlot g_plan_cache[kPlanSlots];

bool same_shape(const ConvShape &a, const ConvShape &b)
{
    return a.c_in == b.c_in && a.h == b.h && a.w == b.w && a.c_out == b.c_out && a.k == b.k &&
           a.stride == b.stride && a.pad == b.pad;
}

int choose_plan(const ConvShape &s, ilpm_plan *p, bool prepacked = false, bool pooled = false)
{
    const int mode = (prepacked ? 1 : 0) | (pooled ? 2 : 0);
    uint64_t h = 1469598103934665603ull;  // FNV-1a over the seven sizes and the mode
    for (int v : {s.c_in, s.h, s.w, s.c_out, s.k, s.stride, s.pad, mode})
        h = (h ^ (uint32_t)v) * 1099511628211ull;
    PlanSlot &slot = g_plan_cache[h % kPlanSlots];
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (slot.used && slot.mode == mode && same_shape(slot.s, s)) {
            *p = slot.p;
            return slot.rc;
        }
    }
    ilpm_plan q = {};
    const int rc = compute_plan(s, &q, prepacked, pooled);
    std::lock_guard<std::mutex> lk(g_mu);
    slot.used = true;
    slot.mode = mode;
    slot.s = s;
    slot.rc = rc;
    slot.p = q;
    *p = q;
    return rc;
}

bool same_plan_shape(const ilpm_plan &a, const ilpm_plan &b)
{
    return a.path == b.path && a.variant == b.variant && a.tile_h == b.tile_h && a.tile_w == b.tile_w &&
           a.co_tile == b.co_tile && a.ci_chunk == b.ci_chunk && a.splits == b.splits && a.grid == b.grid &&
           a.block == b.block && a.lds_bytes == b.lds_bytes && a.h_out == b.h_out && a.w_out == b.w_out &&
           a.workspace_bytes == b.workspace_bytes;
}

// Rebuild the plan the caller passed for this shape and insist it matches, so
// a plan made for another shape is refused rather than run.
int check_plan(const ConvShape &s, const ilpm_plan &p)
{
    ilpm_plan q;
    bool ok = false;
    if (p.path == ILPM_PATH_IGEMM) ok = igemm_make_plan(s, p.variant, p.splits, &q);
    else if (p.path == ILPM_PATH_DIRECT) ok = direct_make_plan(s, p.variant, &q);
    if (!ok || !same_plan_shape(p, q)) return ILPM_ERR_INVALID_ARG;
    return ILPM_OK;
}

// gcnArchName is "gfx950" followed by optional ":feature+/-" settings.
int arch_status(const char *name)
{
    if (!name) return ILPM_ERR_INVALID_ARG;
    return (std::strncmp(name, "gfx950", 6) == 0 && (name[6] == '\0' || name[6] == ':')) ? ILPM_OK : ILPM_ERR_ARCH;
}

int device_check(int *dev_out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return hip_fail(hipErrorInvalidDevice);
    int known = g_arch[dev].load(std::memory_order_acquire);
    if (known == 0) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess) return hip_fail(e);
        known = arch_status(prop.gcnArchName) == ILPM_OK ? 1 : -1;
        g_arch[dev].store(known, std::memory_order_release);
    }
    *dev_out = dev;
    return known == 1 ? ILPM_OK : ILPM_ERR_ARCH;
}

// The workspace of a call on `stream`: the registered one, else the
// library's own, grown when too small.  Growing allocates (hipMalloc) but
// neither synchronises nor frees: the smaller buffer is retired, not freed,
// since work already enqueued or a graph captured earlier may still use it.
// While `stream` is being captured nothing is allocated (an allocation is not
// allowed there): a call that would need to grow returns ILPM_ERR_WORKSPACE.
int get_workspace(int dev, size_t need, hipStream_t stream, void **ws)
{
    *ws = nullptr;
    if (need == 0) return ILPM_OK;
    std::lock_guard<std::mutex> lk(g_mu);
    Workspace &w = g_ws[dev];
    if (w.user) {
        if (w.user_bytes < need) return ILPM_ERR_WORKSPACE;
        *ws = w.user;
        return ILPM_OK;
    }
    if (w.own_bytes < need) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(stream, &cs);
        if (e != hipSuccess) return hip_fail(e);
        if (cs != hipStreamCaptureStatusNone) return ILPM_ERR_WORKSPACE;
        // Geometric growth keeps the retired total below the live buffer.
        size_t bytes = std::max(need, 2 * w.own_bytes);
        bytes = ((bytes + (1u << 20) - 1) >> 20) << 20;
        void *p = nullptr;
        if ((e = hipMalloc(&p, bytes)) != hipSuccess) return hip_fail(e);
        if (w.own) w.retired.push_back(w.own);
        w.own = p;
        w.own_bytes = bytes;
    }
    *ws = w.own;
    return ILPM_OK;
}

// The no-alloc entry point's workspace on device `dev`: the address of that
// device's copy of `scratch`, looked up once per device with the device
// current (the caller's call runs on it).
int scratch_address(int dev, void **ptr)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e);
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return ILPM_OK;
}

void log_plan(const ConvShape &s, const ilpm_plan &p)
{
    static const int on = [] {
        const char *e = std::getenv("ILPM_LOG");
        return e && *e && *e != '0';
    }();
    if (!on) return;
    std::fprintf(stderr,
                 "ilpm: C_in=%d H=%d W=%d C_out=%d K=%d s=%d p=%d -> %s v%d tile %dx%d co%d cc%d splits %d "
                 "grid %d block %d lds %d ws %zu\n",
                 s.c_in, s.h, s.w, s.c_out, s.k, s.stride, s.pad, p.path == ILPM_PATH_IGEMM ? "igemm" : "direct",
                 p.variant, p.tile_h, p.tile_w, p.co_tile, p.ci_chunk, p.splits, p.grid, p.block, p.lds_bytes,
                 p.workspace_bytes);
}

// Workspace bytes a plan needs with an epilogue: the split partial sums, and
// with pooling the full-size conv output (as partial sums for the
// matrix-core path, conv + bias for the direct path).
size_t workspace_need(const ilpm_plan &p, const ConvShape &s, int epilogue)
{
    if (p.path == ILPM_PATH_IGEMM) return igemm_workspace_bytes(p, s, epilogue);
    return (epilogue & ILPM_EPI_MAXPOOL2) ? sizeof(float) * (size_t)s.c_out * s.h_out * s.w_out : 0;
}

// The workspace comes from get_workspace, or with use_scratch from the
// device's fixed `scratch` array (the caller has checked that it is large
// enough).
int run(const float *in, const float *w, const float *bias, const ConvShape &s, float *out, const ilpm_plan &p,
        hipStream_t stream, bool packed = false, int epilogue = 0, bool use_scratch = false)
{
    int dev = 0;
    int rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    void *ws = nullptr;
    const size_t need = workspace_need(p, s, epilogue);
    if (use_scratch) rc = need > 0 ? scratch_address(dev, &ws) : ILPM_OK;
    else rc = get_workspace(dev, need, stream, &ws);
    if (rc != ILPM_OK) return rc;
    log_plan(s, p);
    // Launch errors are read back with hipGetLastError; drop any error an
    // earlier, unrelated runtime call of this thread left behind.
    (void)hipGetLastError();
    hipError_t e;
    const bool relu = (epilogue & ILPM_EPI_RELU) != 0;
    if (p.path == ILPM_PATH_IGEMM) {
        e = igemm_launch(p, s, in, w, bias, out, ws, stream, packed, epilogue);
    } else if (epilogue & ILPM_EPI_MAXPOOL2) {
        float *full = static_cast<float *>(ws);
        e = direct_launch(p, s, in, w, bias, full, stream, false);
        if (e == hipSuccess) e = launch_maxpool2x2(full, s.c_out, s.h_out, s.w_out, out, stream, relu);
    } else {
        e = direct_launch(p, s, in, w, bias, out, stream, relu);
    }
    return e == hipSuccess ? ILPM_OK : hip_fail(e);
}

// Bytes of the prepacked weights of plan p (0 with *rc set on a bad plan).
size_t prepacked_bytes(const ilpm_plan &p, int c_in, int c_out, int k, int *rc)
{
    *rc = ILPM_OK;
    if (c_in <= 0 || c_out <= 0 || k <= 0 || (int64_t)c_out * c_in * k * k > kMaxElems) {
        *rc = ILPM_ERR_INVALID_ARG;
        return 0;
    }
    int kk = 0, st = 0, th, tw, ct;
    if (p.path == ILPM_PATH_IGEMM) {
        if (!igemm_variant_info(p.variant, &kk, &st, &th, &tw, &ct) || kk != k) {
            *rc = ILPM_ERR_INVALID_ARG;
            return 0;
        }
        return sizeof(float) * (size_t)igemm_packed_floats(p, c_in, c_out);
    }
    if (p.path == ILPM_PATH_DIRECT && p.variant >= 0 && p.variant < direct_num_variants())
        return sizeof(float) * (size_t)c_out * c_in * k * k;
    *rc = ILPM_ERR_INVALID_ARG;
    return 0;
}

}  // namespace
}  // namespace ilpm

using namespace ilpm;

extern "C" {

const char *ilpm_status_str(int status)
{
    switch (status) {
    case ILPM_OK: return "ok";
    case ILPM_ERR_INVALID_ARG: return "invalid argument";
    case ILPM_ERR_UNSUPPORTED: return "unsupported size";
    case ILPM_ERR_WORKSPACE: return "workspace too small";
    case ILPM_ERR_HIP: return "HIP runtime error";
    case ILPM_ERR_ARCH: return "device is not gfx950";
    default: return "unknown status";
    }
}

int ilpm_conv2d_validate(const void *in, const void *w, const void *bias, int C_in, int H, int W, int C_out,
                         int K, int stride, int pad, const void *out)
{
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    return validate(in, w, bias, s, out);
}

int ilpm_conv2d_plan(int C_in, int H, int W, int C_out, int K, int stride, int pad, ilpm_plan *plan)
{
    if (!plan) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    return choose_plan(s, plan);
}

int ilpm_conv2d_plan_prepacked(int C_in, int H, int W, int C_out, int K, int stride, int pad, ilpm_plan *plan)
{
    if (!plan) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    return choose_plan(s, plan, true);
}

int ilpm_conv2d_plan_for(int C_in, int H, int W, int C_out, int K, int stride, int pad, int epilogue,
                         int prepacked, ilpm_plan *plan)
{
    if (!plan || (epilogue & ~(ILPM_EPI_RELU | ILPM_EPI_MAXPOOL2)) || (prepacked != 0 && prepacked != 1))
        return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    return choose_plan(s, plan, prepacked != 0, (epilogue & ILPM_EPI_MAXPOOL2) != 0);
}

int ilpm_conv2d_plan_variant(int C_in, int H, int W, int C_out, int K, int stride, int pad, int path,
                             int variant, int splits, ilpm_plan *plan)
{
    if (!plan) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    bool ok = false;
    if (path == ILPM_PATH_IGEMM) ok = igemm_make_plan(s, variant, splits, plan);
    else if (path == ILPM_PATH_DIRECT) ok = splits <= 1 && direct_make_plan(s, variant, plan);
    return ok ? ILPM_OK : ILPM_ERR_INVALID_ARG;
}

const char *ilpm_variant_name(int path, int variant)
{
    if (path == ILPM_PATH_IGEMM) return igemm_variant_name(variant);
    if (path == ILPM_PATH_DIRECT) return direct_variant_name(variant);
    return nullptr;
}

int ilpm_num_variants(int path)
{
    if (path == ILPM_PATH_IGEMM) return igemm_num_variants();
    if (path == ILPM_PATH_DIRECT) return direct_num_variants();
    return 0;
}

int ilpm_variant_info(int path, int variant, int *K, int *stride, int *tile_h, int *tile_w, int *co_tile)
{
    int k, st, th, tw, ct;
    bool ok = false;
    if (path == ILPM_PATH_IGEMM) ok = igemm_variant_info(variant, &k, &st, &th, &tw, &ct);
    else if (path == ILPM_PATH_DIRECT) ok = direct_variant_info(variant, &k, &st, &th, &tw, &ct);
    if (!ok) return ILPM_ERR_INVALID_ARG;
    if (K) *K = k;
    if (stride) *stride = st;
    if (tile_h) *tile_h = th;
    if (tile_w) *tile_w = tw;
    if (co_tile) *co_tile = ct;
    return ILPM_OK;
}

int ilpm_variant_pipeline(int path, int variant, int *ci_chunk, int *stages, int *buffers, int *flags)
{
    int cc = 0, ns = 0, nb = 0, fl = 0;
    if (path == ILPM_PATH_IGEMM) {
        if (!igemm_variant_pipeline(variant, &cc, &ns, &nb, &fl)) return ILPM_ERR_INVALID_ARG;
    } else if (path != ILPM_PATH_DIRECT || variant < 0 || variant >= direct_num_variants()) {
        return ILPM_ERR_INVALID_ARG;
    }
    if (ci_chunk) *ci_chunk = cc;
    if (stages) *stages = ns;
    if (buffers) *buffers = nb;
    if (flags) *flags = fl;
    return ILPM_OK;
}

int ilpm_conv2d_workspace_size(int C_in, int H, int W, int C_out, int K, int stride, int pad, size_t *bytes)
{
    if (!bytes) return ILPM_ERR_INVALID_ARG;
    ilpm_plan p;
    int rc = ilpm_conv2d_plan(C_in, H, W, C_out, K, stride, pad, &p);
    if (rc != ILPM_OK) return rc;
    *bytes = p.workspace_bytes;
    return ILPM_OK;
}

int ilpm_conv2d_epilogue_workspace_size(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                                        int epilogue, const ilpm_plan *plan, size_t *bytes)
{
    if (!bytes || (epilogue & ~(ILPM_EPI_RELU | ILPM_EPI_MAXPOOL2))) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    ilpm_plan p;
    if (plan) {
        rc = check_plan(s, *plan);
        p = *plan;
    } else {
        rc = choose_plan(s, &p, false, (epilogue & ILPM_EPI_MAXPOOL2) != 0);
    }
    if (rc != ILPM_OK) return rc;
    *bytes = workspace_need(p, s, epilogue);
    return ILPM_OK;
}

int ilpm_last_hip_error(void) { return g_last_hip; }

int ilpm_set_split_sum(int mode) { return igemm_set_split_sum(mode) ? ILPM_OK : ILPM_ERR_INVALID_ARG; }

int ilpm_set_workspace(void *ptr, size_t bytes, hipStream_t stream)
{
    (void)stream;
    if (ptr && ((uintptr_t)ptr & 255u)) return ILPM_ERR_INVALID_ARG;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return hip_fail(hipErrorInvalidDevice);
    std::lock_guard<std::mutex> lk(g_mu);
    g_ws[dev].user = ptr;
    g_ws[dev].user_bytes = ptr ? bytes : 0;
    return ILPM_OK;
}

int ilpm_conv2d_fwd(const float *in, const float *w, const float *bias, int C_in, int H, int W, int C_out, int K,
                    int stride, int pad, float *out, hipStream_t stream)
{
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    rc = validate(in, w, bias, s, out);
    if (rc != ILPM_OK) return rc;
    ilpm_plan p;
    rc = choose_plan(s, &p);
    if (rc != ILPM_OK) return rc;
    return run(in, w, bias, s, out, p, stream);
}

int ilpm_arch_supported(const char *gcn_arch_name) { return arch_status(gcn_arch_name); }

int ilpm_conv2d_fwd_noalloc(const float *in, const float *w, const float *bias, int C_in, int H, int W, int C_out,
                            int K, int stride, int pad, float *out, hipStream_t stream)
{
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    rc = validate(in, w, bias, s, out);
    if (rc != ILPM_OK) return rc;
    ilpm_plan p;
    rc = choose_plan(s, &p);
    if (rc != ILPM_OK) return rc;
    if (workspace_need(p, s, 0) > ILPM_NOALLOC_SCRATCH_BYTES) return ILPM_ERR_WORKSPACE;
    return run(in, w, bias, s, out, p, stream, false, 0, true);
}

int ilpm_conv2d_fwd_plan(const float *in, const float *w, const float *bias, int C_in, int H, int W, int C_out,
                         int K, int stride, int pad, float *out, const ilpm_plan *plan, hipStream_t stream)
{
    if (!plan) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    rc = validate(in, w, bias, s, out);
    if (rc != ILPM_OK) return rc;
    rc = check_plan(s, *plan);
    if (rc != ILPM_OK) return rc;
    return run(in, w, bias, s, out, *plan, stream);
}

int ilpm_conv2d_prepacked_size(const ilpm_plan *plan, int C_in, int C_out, int K, size_t *bytes)
{
    if (!plan || !bytes) return ILPM_ERR_INVALID_ARG;
    int rc;
    const size_t b = prepacked_bytes(*plan, C_in, C_out, K, &rc);
    if (rc != ILPM_OK) return rc;
    *bytes = b;
    return ILPM_OK;
}

int ilpm_conv2d_prepack_weights(const float *w, int C_in, int C_out, int K, const ilpm_plan *plan, float *packed,
                                hipStream_t stream)
{
    if (!plan || !w || !packed) return ILPM_ERR_INVALID_ARG;
    int rc;
    const size_t pb = prepacked_bytes(*plan, C_in, C_out, K, &rc);
    if (rc != ILPM_OK) return rc;
    if (((uintptr_t)w | (uintptr_t)packed) & 15u) return ILPM_ERR_INVALID_ARG;
    if (overlaps(w, sizeof(float) * (size_t)C_out * C_in * K * K, packed, pb)) return ILPM_ERR_INVALID_ARG;
    int dev = 0;
    rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    (void)hipGetLastError();
    hipError_t e;
    if (plan->path == ILPM_PATH_IGEMM) e = igemm_pack(*plan, C_in, C_out, w, packed, stream);
    else e = hipMemcpyAsync(packed, w, pb, hipMemcpyDeviceToDevice, stream);
    return e == hipSuccess ? ILPM_OK : hip_fail(e);
}

int ilpm_conv2d_fwd_prepacked(const float *in, const float *packed, const float *bias, int C_in, int H, int W,
                              int C_out, int K, int stride, int pad, const ilpm_plan *plan, float *out,
                              hipStream_t stream)
{
    if (!plan || !packed) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    // The OIHW-size checks of validate() cover in, bias and out; the packed
    // buffer gets its own size.
    rc = validate(in, packed, bias, s, out);
    if (rc != ILPM_OK) return rc;
    const size_t pb = prepacked_bytes(*plan, C_in, C_out, K, &rc);
    if (rc != ILPM_OK) return rc;
    if (((uintptr_t)packed & 15u) || overlaps(out, sizeof(float) * (size_t)C_out * s.h_out * s.w_out, packed, pb))
        return ILPM_ERR_INVALID_ARG;
    rc = check_plan(s, *plan);
    if (rc != ILPM_OK) return rc;
    return run(in, packed, bias, s, out, *plan, stream, true);
}

int ilpm_conv2d_fwd_prepacked_epilogue(const float *in, const float *packed, const float *bias, int C_in, int H,
                                       int W, int C_out, int K, int stride, int pad, int epilogue,
                                       const ilpm_plan *plan, float *out, hipStream_t stream)
{
    if (!plan || !packed || (epilogue & ~(ILPM_EPI_RELU | ILPM_EPI_MAXPOOL2))) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    if ((epilogue & ILPM_EPI_MAXPOOL2) && (s.h_out < 2 || s.w_out < 2)) return ILPM_ERR_INVALID_ARG;
    rc = validate(in, packed, bias, s, out, epilogue);
    if (rc != ILPM_OK) return rc;
    const size_t pb = prepacked_bytes(*plan, C_in, C_out, K, &rc);
    if (rc != ILPM_OK) return rc;
    if (((uintptr_t)packed & 15u) || overlaps(out, out_bytes(s, epilogue), packed, pb))
        return ILPM_ERR_INVALID_ARG;
    rc = check_plan(s, *plan);
    if (rc != ILPM_OK) return rc;
    return run(in, packed, bias, s, out, *plan, stream, true, epilogue);
}

int ilpm_conv2d_fwd_epilogue(const float *in, const float *w, const float *bias, int C_in, int H, int W, int C_out,
                             int K, int stride, int pad, int epilogue, const ilpm_plan *plan, float *out,
                             hipStream_t stream)
{
    if (epilogue & ~(ILPM_EPI_RELU | ILPM_EPI_MAXPOOL2)) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, K, stride, pad, &s);
    if (rc != ILPM_OK) return rc;
    if ((epilogue & ILPM_EPI_MAXPOOL2) && (s.h_out < 2 || s.w_out < 2)) return ILPM_ERR_INVALID_ARG;
    rc = validate(in, w, bias, s, out, epilogue);
    if (rc != ILPM_OK) return rc;
    ilpm_plan p;
    if (plan) {
        rc = check_plan(s, *plan);
        p = *plan;
    } else {
        rc = choose_plan(s, &p, false, (epilogue & ILPM_EPI_MAXPOOL2) != 0);
    }
    if (rc != ILPM_OK) return rc;
    return run(in, w, bias, s, out, p, stream, false, epilogue);
}

int ilpm_winograd_filter_size(int C_in, int C_out, size_t *bytes)
{
    if (!bytes || C_in <= 0 || C_out <= 0 || (int64_t)C_out * C_in * 16 > kMaxElems) return ILPM_ERR_INVALID_ARG;
    *bytes = sizeof(float) * 16 * (size_t)C_out * C_in;
    return ILPM_OK;
}

int ilpm_winograd_transform_filter(const float *w, int C_in, int C_out, float *u, hipStream_t stream)
{
    size_t ub = 0;
    int rc = ilpm_winograd_filter_size(C_in, C_out, &ub);
    if (rc != ILPM_OK) return rc;
    if (!w || !u || (((uintptr_t)w | (uintptr_t)u) & 3u)) return ILPM_ERR_INVALID_ARG;
    if (overlaps(w, sizeof(float) * 9 * (size_t)C_out * C_in, u, ub)) return ILPM_ERR_INVALID_ARG;
    int dev = 0;
    rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    (void)hipGetLastError();
    const hipError_t e = winograd_filter_launch(w, C_in, C_out, u, stream);
    return e == hipSuccess ? ILPM_OK : hip_fail(e);
}

int ilpm_conv2d_winograd_workspace_size(int C_in, int H, int W, int C_out, int pad, size_t *bytes)
{
    if (!bytes) return ILPM_ERR_INVALID_ARG;
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, 3, 1, pad, &s);
    if (rc != ILPM_OK) return rc;
    *bytes = winograd_workspace_bytes(s);
    return ILPM_OK;
}

int ilpm_conv2d_fwd_winograd(const float *in, const float *u, const float *bias, int C_in, int H, int W, int C_out,
                             int pad, float *out, hipStream_t stream)
{
    ConvShape s;
    int rc = check_dims(C_in, H, W, C_out, 3, 1, pad, &s);
    if (rc != ILPM_OK) return rc;
    if (!in || !u || !out) return ILPM_ERR_INVALID_ARG;
    if (((uintptr_t)in | (uintptr_t)u | (uintptr_t)out | (uintptr_t)bias) & 3u) return ILPM_ERR_INVALID_ARG;
    const size_t in_b = sizeof(float) * (size_t)C_in * H * W, u_b = sizeof(float) * 16 * (size_t)C_out * C_in;
    const size_t o_b = sizeof(float) * (size_t)C_out * s.h_out * s.w_out, b_b = sizeof(float) * (size_t)C_out;
    if (overlaps(out, o_b, in, in_b) || overlaps(out, o_b, u, u_b) || overlaps(out, o_b, bias, b_b))
        return ILPM_ERR_INVALID_ARG;
    // Offsets and the library GEMM's sizes are 32-bit.
    const int64_t t = winograd_tiles(s);
    if (16 * (int64_t)C_in * t > kMaxElems || 16 * (int64_t)C_out * t > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    int dev = 0;
    rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    void *ws = nullptr;
    rc = get_workspace(dev, winograd_workspace_bytes(s), stream, &ws);
    if (rc != ILPM_OK) return rc;
    (void)hipGetLastError();
    hipError_t e;
    rc = winograd_launch(s, in, u, bias, out, ws, dev, stream, &e);
    if (rc == ILPM_ERR_HIP && e != hipSuccess) return hip_fail(e);
    return rc;
}

int ilpm_relu_inplace(float *x, int64_t n, hipStream_t stream)
{
    if (n < 0 || (!x && n > 0) || ((uintptr_t)x & 3u)) return ILPM_ERR_INVALID_ARG;
    if (n == 0) return ILPM_OK;
    int dev = 0;
    int rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    (void)hipGetLastError();
    const hipError_t e = launch_relu(x, n, stream);
    return e == hipSuccess ? ILPM_OK : hip_fail(e);
}

int ilpm_maxpool2x2(const float *in, int C, int H, int W, float *out, hipStream_t stream)
{
    if (!in || !out || C <= 0 || H < 2 || W < 2) return ILPM_ERR_INVALID_ARG;
    if ((int64_t)C * H * W > kMaxElems) return ILPM_ERR_UNSUPPORTED;
    if (((uintptr_t)in | (uintptr_t)out) & 3u) return ILPM_ERR_INVALID_ARG;
    const size_t in_b = sizeof(float) * (size_t)C * H * W;
    const size_t o_b = sizeof(float) * (size_t)C * (H / 2) * (W / 2);
    if (overlaps(in, in_b, out, o_b)) return ILPM_ERR_INVALID_ARG;
    int dev = 0;
    int rc = device_check(&dev);
    if (rc != ILPM_OK) return rc;
    (void)hipGetLastError();
    const hipError_t e = launch_maxpool2x2(in, C, H, W, out, stream, false);
    return e == hipSuccess ? ILPM_OK : hip_fail(e);
}

}  // extern "C"

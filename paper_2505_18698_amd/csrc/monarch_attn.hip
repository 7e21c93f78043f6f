// C ABI of the MonarchAttention forward pass (include/monarch_attn.h):
// argument checks, the per-device workspace, path selection and per-launch
// timing.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <unordered_map>
#include <vector>

#include "host_common.hpp"

namespace ma_host {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

Timing g_timing;

}  // namespace ma_host

namespace {

using namespace ma_host;

size_t elem_bytes(int32_t dtype) { return dtype == MA_F32 ? 4 : 2; }

int check_shape(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    if (dtype != MA_F32 && dtype != MA_BF16 && dtype != MA_F16) return fail(MA_EINVAL, "unknown dtype %d", dtype);
    if (b < 1 || d < 1 || N < 0 || m < 0) return fail(MA_EINVAL, "N, m must be >= 0 and d, b >= 1");
    if (N == 0 ? m != 0 : (m < 1 || N > m * b || N <= (m - 1) * b))
        return fail(MA_EINVAL, "m (%lld) must be ceil(N / b) (N = %lld, b = %lld)", (long long)m, (long long)N,
                    (long long)b);
    if (T < 1) return fail(MA_EINVAL, "T must be >= 1 (got %d)", T);
    if (T > 64) return fail(MA_EUNSUPPORTED, "T > 64 is not supported (got %d)", T);
    if (dtype != MA_F32 && T > MONARCH_ATTN_MAX_T_16BIT)
        return fail(MA_EUNSUPPORTED,
                    "bf16 and fp16 take T <= %d, the step count up to which their accuracy is validated (got %d)",
                    MONARCH_ATTN_MAX_T_16BIT, T);
    if (m > 128 || b > 128) return fail(MA_EUNSUPPORTED, "m and b must be <= 128 (got m=%lld, b=%lld)", (long long)m, (long long)b);
    // rows of 16-byte multiples (so every row of q, k, v, out is 16-byte aligned), at most 128 wide
    if (d > 128 || d % (16 / (int64_t)elem_bytes(dtype)) != 0)
        return fail(MA_EUNSUPPORTED, "d must be a multiple of %d up to 128 (got %lld)", (int)(16 / elem_bytes(dtype)),
                    (long long)d);
    // fp32 tiles of the half-steps: tile rows (16, 32, 64 or 128) times D at most 8192 elements
    const int64_t D = tile_d(d);
    if (dtype == MA_F32 && ((int64_t)tile_rows(m) * D > 8192 || (int64_t)tile_rows(b) * D > 8192))
        return fail(MA_EUNSUPPORTED, "fp32 needs tile(m)*D <= 8192 and tile(b)*D <= 8192 (tile: 16, 32, 64 or 128 "
                    "rows, D = %lld)", (long long)D);
    return MA_OK;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Np = m * b: the states cover the padded sequence, with rows of d elements.
size_t state_bytes(int64_t BH, int64_t Np, int64_t d, int32_t dtype)
{
    return align_up((size_t)BH * Np * d * elem_bytes(dtype));
}

size_t workspace_bytes(int64_t BH, int64_t Np, int64_t d, int32_t dtype)
{
    // alpha_R, alpha_L and Y in the element type, c_R and c_L in fp32
    const size_t st = state_bytes(BH, Np, d, dtype);
    const size_t cs = align_up((size_t)BH * Np * sizeof(float));
    return 3 * st + 2 * cs;
}

// The workspace of one (device, stream): calls on one stream are ordered by
// it, so they can share one; calls on different streams get their own.  `mu`
// is held by a call from acquiring the workspace to its last launch, so that
// the launches of two calls on one stream never interleave.
struct Workspace {
    std::mutex mu;
    void *ptr = nullptr;
    size_t bytes = 0;
    // A call captured into a HIP graph bakes `ptr` into the graph, so a
    // buffer that was ever used under capture is not freed when the
    // workspace grows: it is kept in `retired` until
    // monarch_attn_release_workspace.
    bool captured = false;
    std::vector<void *> retired;
};

// The scratch of monarch_attn_fwd_noalloc: the states of the half-step path,
// one array per device for the life of the process.  In host code `scratch`
// names a host-side stand-in: its device address comes from
// hipGetSymbolAddress (Device::scratch), once per device.
static __device__ __align__(256) unsigned char scratch[MONARCH_ATTN_NOALLOC_SCRATCH_BYTES];

struct Device {
    void *scratch = nullptr;  // device address of `scratch` on this device (null: not looked up yet)
    int num_cus = 0;  // 0: not queried yet
    // Entries are never erased (a caller may be waiting on an entry's mutex);
    // release only frees their memory.
    std::unordered_map<hipStream_t, std::unique_ptr<Workspace>> ws;
};

constexpr int kMaxDevices = 64;
std::mutex g_dev_mutex;
Device g_dev[kMaxDevices];
std::atomic<int> g_path{kAuto};
std::mutex g_timing_mutex;

bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// B * H heads of `per` workgroups each must fit one grid (fewer than 2^31
// workgroups), checked without forming a product that could overflow.
int check_heads(int64_t B, int64_t H, int64_t per)
{
    if (B < 0 || H < 0) return fail(MA_EINVAL, "B and H must be >= 0");
    const int64_t lim = (int64_t)0x7fffffff / (per > 0 ? per : 1);
    if (B > lim || H > lim || (H > 0 && B > lim / H)) return fail(MA_EUNSUPPORTED, "too many heads for one grid");
    return MA_OK;
}

// The current device and its compute-unit count (queried once per device).
int current_device(int &dev, int &num_cus)
{
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return fail(MA_EHIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> lock(g_dev_mutex);
    Device &D = g_dev[dev];
    if (D.num_cus == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
            return fail(MA_EHIP, "querying the compute unit count failed");
        D.num_cus = n;
    }
    num_cus = D.num_cus;
    return MA_OK;
}

// The device address of the no-allocation scratch on device `dev` (the
// current device), looked up on its first use there.
int noalloc_scratch(int dev, char **base)
{
    std::lock_guard<std::mutex> lock(g_dev_mutex);
    Device &D = g_dev[dev];
    if (!D.scratch) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(MA_EHIP, "hipGetSymbolAddress of the scratch array failed: %s", hipGetErrorString(e));
        }
        D.scratch = p;
    }
    *base = (char *)D.scratch;
    return MA_OK;
}

// Whether `stream` is being captured into a HIP graph.
int stream_capturing(hipStream_t stream, bool &capturing)
{
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &st) != hipSuccess) {
        (void)hipGetLastError();
        return fail(MA_EHIP, "hipStreamIsCapturing failed");
    }
    capturing = st != hipStreamCaptureStatusNone;
    return MA_OK;
}

// The workspace of (dev, stream), locked into `hold` for the caller and grown
// with hipMalloc to at least `need` bytes.  Growing first waits for the
// stream, whose earlier calls may still use the old buffer.  A stream under
// graph capture cannot allocate or wait: its workspace must already be
// large enough.  The first call not under capture after a capture moves to a
// fresh buffer: a graph replays on whatever stream its caller picks, so it
// must not share its buffer with the eager calls on the capture stream.
int acquire_workspace(int dev, hipStream_t stream, bool capturing, size_t need, char **base,
                      std::unique_lock<std::mutex> &hold)
{
    Workspace *w;
    {
        std::lock_guard<std::mutex> lock(g_dev_mutex);
        std::unique_ptr<Workspace> &slot = g_dev[dev].ws[stream];
        if (!slot) slot.reset(new Workspace);
        w = slot.get();
    }
    hold = std::unique_lock<std::mutex>(w->mu);
    if (w->bytes < need || (w->captured && !capturing)) {
        if (capturing)
            return fail(MA_EUNSUPPORTED,
                        "the stream is being captured and its workspace holds %zu of the %zu bytes this call needs: "
                        "make a call of this size on the stream before capturing",
                        w->bytes, need);
        if (w->bytes > need) need = w->bytes;  // a move off a captured buffer keeps its size
        if (w->ptr) {
            if (w->captured) {
                w->retired.push_back(w->ptr);  // a captured graph may still use it
            } else {
                if (hipStreamSynchronize(stream) != hipSuccess) return fail(MA_EHIP, "hipStreamSynchronize failed");
                (void)hipFree(w->ptr);
            }
            w->ptr = nullptr;
            w->bytes = 0;
            w->captured = false;
        }
        void *p = nullptr;
        if (hipMalloc(&p, need) != hipSuccess) {
            (void)hipGetLastError();
            return fail(MA_ENOMEM, "hipMalloc of %zu workspace bytes failed", need);
        }
        w->ptr = p;
        w->bytes = need;
    }
    if (capturing) w->captured = true;
    *base = (char *)w->ptr;
    return MA_OK;
}

// Per-launch timing records events, which a graph capture would take in.
int check_capture(hipStream_t stream, bool &capturing)
{
    int rc = stream_capturing(stream, capturing);
    if (rc != MA_OK) return rc;
    if (capturing && g_timing.enabled) return fail(MA_EUNSUPPORTED, "per-launch timing is on: it cannot be captured");
    return MA_OK;
}

// The forward pass; with obj != nullptr also the objective per (head, step);
// with need_lens, per-sequence lengths lens[B] (device).
// noalloc: the states go to the scratch array instead of the stream's
// workspace (no objective, no lengths).  prepad: pre-padded sequences.
int forward(const void *q, const void *k, const void *v, void *out, float *obj, bool need_obj, const int32_t *lens,
            bool need_lens, int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype,
            void *stream, bool noalloc = false, bool prepad = false)
{
    g_err[0] = '\0';
    if (B < 0 || H < 0) return fail(MA_EINVAL, "B and H must be >= 0");
    int rc = check_shape(N, d, m, b, T, dtype);
    if (rc != MA_OK) return rc;
    if ((rc = check_heads(B, H, m > b ? m : b)) != MA_OK) return rc;
    if (B == 0 || H == 0 || N == 0) return MA_OK;  // nothing to compute: no launch, no pointer read
    if (!q || !k || !v || !out) return fail(MA_EINVAL, "null tensor pointer");
    if (need_obj && !obj) return fail(MA_EINVAL, "null objective pointer");
    if (need_obj && ((uintptr_t)obj & 3u)) return fail(MA_EINVAL, "obj must be 4-byte aligned");
    if (need_lens && !lens) return fail(MA_EINVAL, "null lens pointer");
    if (need_lens && ((uintptr_t)lens & 3u)) return fail(MA_EINVAL, "lens must be 4-byte aligned");
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)out) & 15u)
        return fail(MA_EINVAL, "q, k, v and out must be 16-byte aligned");
    const int64_t BH = B * H;
    const size_t tensor_bytes = (size_t)BH * N * d * elem_bytes(dtype);
    if (overlaps(out, tensor_bytes, q, tensor_bytes) || overlaps(out, tensor_bytes, k, tensor_bytes) ||
        overlaps(out, tensor_bytes, v, tensor_bytes))
        return fail(MA_EINVAL, "out must not overlap q, k or v");
    const size_t obj_bytes = (size_t)BH * T * sizeof(float);
    if (obj && (overlaps(obj, obj_bytes, q, tensor_bytes) || overlaps(obj, obj_bytes, k, tensor_bytes) ||
                overlaps(obj, obj_bytes, v, tensor_bytes) || overlaps(obj, obj_bytes, out, tensor_bytes)))
        return fail(MA_EINVAL, "obj must not overlap q, k, v or out");
    if (lens && overlaps(lens, (size_t)B * sizeof(int32_t), out, tensor_bytes))
        return fail(MA_EINVAL, "lens must not overlap out");

    const int path = g_path.load();
    const size_t st = state_bytes(BH, m * b, d, dtype);
    const size_t cs = align_up((size_t)BH * m * b * sizeof(float));
    CallBufs bufs{q, k, v, out, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, obj, lens, prepad ? 1 : 0};
    int dev = 0, num_cus = 0;
    if ((rc = current_device(dev, num_cus)) != MA_OK) return rc;
    bool capturing = false;
    if ((rc = check_capture((hipStream_t)stream, capturing)) != MA_OK) return rc;
    std::unique_lock<std::mutex> ws_hold;  // the stream's workspace, held until the launches are enqueued
    const int fam = family_of(path, dtype, d, m, b, need_lens || prepad, need_obj);
    const bool states = fam == kFamHalf;  // the other families keep their states in LDS
    const size_t obj_part_bytes = obj ? align_up((size_t)BH * T * b * sizeof(float)) : 0;
    if (states || obj) {
        const size_t state_ws = states ? workspace_bytes(BH, m * b, d, dtype) : 0;
        char *base = nullptr;
        if (noalloc) {
            if (state_ws + obj_part_bytes > MONARCH_ATTN_NOALLOC_SCRATCH_BYTES)
                return fail(MA_EUNSUPPORTED,
                            "the states of this call take %zu bytes, more than the %llu bytes of the no-allocation "
                            "scratch",
                            state_ws + obj_part_bytes, (unsigned long long)MONARCH_ATTN_NOALLOC_SCRATCH_BYTES);
            if ((rc = noalloc_scratch(dev, &base)) != MA_OK) return rc;
        } else if ((rc = acquire_workspace(dev, (hipStream_t)stream, capturing, state_ws + obj_part_bytes, &base,
                                           ws_hold)) != MA_OK) {
            return rc;
        }
        if (states) {
            bufs.aR = base;
            bufs.aL = base + st;
            bufs.Y = base + 2 * st;
            bufs.cR = (float *)(base + 3 * st);
            bufs.cL = (float *)(base + 3 * st + cs);
        }
        if (obj) bufs.obj_part = (float *)(base + state_ws);
    }
    CallDims dims{BH, H, (int)m, (int)b, (int)N, (int)d, T, (float)(1.4426950408889634 / std::sqrt((double)d)),
                  num_cus};

    std::unique_lock<std::mutex> tlock(g_timing_mutex);
    Launcher L{(hipStream_t)stream, g_timing.enabled};
    if (!L.timed) tlock.unlock();
    (void)hipGetLastError();  // clear a stale error so the check below is ours
    switch (dtype) {
    case MA_F32: rc = run_call<float>(L, bufs, dims, path); break;
    case MA_BF16: rc = run_call<__bf16>(L, bufs, dims, path); break;
    default: rc = run_call<_Float16>(L, bufs, dims, path); break;
    }
    if (L.timed) {
        g_timing.nlaunch = L.n;
        g_timing.ready = (rc == MA_OK && L.n > 0);
    }
    if (rc != MA_OK) return rc;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(MA_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MA_OK;
}

// ---- gradient ----

// The gradient takes every shape the forward takes (its 128-row units at
// D = 128 hold the tiles that are exact in the 16-bit element type as such),
// for T <= 32.
int check_bwd_shape(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    const int rc = check_shape(N, d, m, b, T, dtype);
    if (rc != MA_OK) return rc;
    if (T > 32) return fail(MA_EUNSUPPORTED, "the gradient supports T <= 32 (got %d)", T);
    if (dtype != MA_F32 && T > MONARCH_ATTN_MAX_T_16BIT_BWD)
        return fail(MA_EUNSUPPORTED,
                    "the gradient in bf16 and fp16 takes T <= %d, the step count up to which its accuracy is "
                    "validated (got %d)",
                    MONARCH_ATTN_MAX_T_16BIT_BWD, T);
    return MA_OK;
}

// Workspace of one gradient call, in this order: alpha_R of steps 2..T, alpha_L
// of steps 1..T and Y (element type, rows of d elements); c_R of steps
// 2..T and c_L of steps 1..T (fp32); the fp32 accumulators of dQ and dK
// ([B*H][N][d]); the fp32 gradients d alpha_L, dY, d alpha_R (width D) and
// d c_L, d c_R.
struct BwdLayout {
    size_t st, cs, acc, sg;
    int32_t T;
    size_t states() const { return (size_t)(2 * T) * st + (size_t)(2 * T - 1) * cs; }
    size_t total() const { return states() + 2 * acc + 3 * sg + 2 * cs; }
};

BwdLayout bwd_layout(int64_t BH, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    const int64_t Np = m * b;
    return BwdLayout{state_bytes(BH, Np, d, dtype), align_up((size_t)BH * Np * sizeof(float)),
                     align_up((size_t)BH * N * d * sizeof(float)), align_up((size_t)BH * Np * tile_d(d) * sizeof(float)),
                     T};
}

int backward(const void *q, const void *k, const void *v, const void *dout, void *dq, void *dk, void *dv,
             const int32_t *lens, bool need_lens, int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b,
             int32_t T, int32_t dtype, void *stream)
{
    g_err[0] = '\0';
    if (B < 0 || H < 0) return fail(MA_EINVAL, "B and H must be >= 0");
    int rc = check_bwd_shape(N, d, m, b, T, dtype);
    if (rc != MA_OK) return rc;
    if ((rc = check_heads(B, H, m > b ? m : b)) != MA_OK) return rc;
    if (B == 0 || H == 0 || N == 0) return MA_OK;  // nothing to compute: no launch, no pointer read
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return fail(MA_EINVAL, "null tensor pointer");
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)dout | (uintptr_t)dq | (uintptr_t)dk |
         (uintptr_t)dv) & 15u)
        return fail(MA_EINVAL, "all tensors must be 16-byte aligned");
    if (need_lens && !lens) return fail(MA_EINVAL, "null lens pointer");
    if (need_lens && ((uintptr_t)lens & 3u)) return fail(MA_EINVAL, "lens must be 4-byte aligned");
    const int64_t BH = B * H;
    const size_t tb = (size_t)BH * N * d * elem_bytes(dtype);
    const void *ins[4] = {q, k, v, dout};
    void *outs[3] = {dq, dk, dv};
    for (int o = 0; o < 3; ++o) {
        for (int i = 0; i < 4; ++i)
            if (overlaps(outs[o], tb, ins[i], tb)) return fail(MA_EINVAL, "dq, dk, dv must not overlap q, k, v or dout");
        for (int o2 = o + 1; o2 < 3; ++o2)
            if (overlaps(outs[o], tb, outs[o2], tb)) return fail(MA_EINVAL, "dq, dk and dv must not overlap");
        if (lens && overlaps(outs[o], tb, lens, (size_t)B * sizeof(int32_t)))
            return fail(MA_EINVAL, "lens must not overlap dq, dk or dv");
    }
    int dev = 0, num_cus = 0;
    if ((rc = current_device(dev, num_cus)) != MA_OK) return rc;
    bool capturing = false;
    if ((rc = check_capture((hipStream_t)stream, capturing)) != MA_OK) return rc;
    const BwdLayout lay = bwd_layout(BH, N, d, m, b, T, dtype);
    char *base = nullptr;
    std::unique_lock<std::mutex> ws_hold;  // the stream's workspace, held until the launches are enqueued
    if ((rc = acquire_workspace(dev, (hipStream_t)stream, capturing, lay.total(), &base, ws_hold)) != MA_OK)
        return rc;
    BwdCallBufs bufs{};
    bufs.q = q, bufs.k = k, bufs.v = v, bufs.dout = dout, bufs.dq = dq, bufs.dk = dk, bufs.dv = dv;
    bufs.lens = lens;
    char *p = base;
    bufs.st = lay.st;
    bufs.cst = lay.cs / sizeof(float);
    bufs.aR = p, p += (size_t)(T - 1) * lay.st;
    bufs.aL = p, p += (size_t)T * lay.st;
    bufs.Y = p, p += lay.st;
    bufs.cR = (float *)p, p += (size_t)(T - 1) * lay.cs;
    bufs.cL = (float *)p, p += (size_t)T * lay.cs;
    bufs.dQ = (float *)p, p += lay.acc;
    bufs.dK = (float *)p, p += lay.acc;
    bufs.daL = (float *)p, p += lay.sg;
    bufs.dY = (float *)p, p += lay.sg;
    bufs.daR = (float *)p, p += lay.sg;
    bufs.dcL = (float *)p, p += lay.cs;
    bufs.dcR = (float *)p;
    CallDims dims{BH, H, (int)m, (int)b, (int)N, (int)d, T, (float)(1.4426950408889634 / std::sqrt((double)d)),
                  num_cus};

    std::unique_lock<std::mutex> tlock(g_timing_mutex);
    Launcher L{(hipStream_t)stream, g_timing.enabled};
    if (!L.timed) tlock.unlock();
    (void)hipGetLastError();
    switch (dtype) {
    case MA_F32: rc = run_bwd<float>(L, bufs, dims); break;
    case MA_BF16: rc = run_bwd<__bf16>(L, bufs, dims); break;
    default: rc = run_bwd<_Float16>(L, bufs, dims); break;
    }
    if (L.timed) {
        g_timing.nlaunch = L.n;
        g_timing.ready = (rc == MA_OK && L.n > 0);
    }
    if (rc != MA_OK) return rc;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(MA_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MA_OK;
}

}  // namespace

#ifndef MA_BUILD_ID
#error "MA_BUILD_ID (the source hash) is defined by paper_2505_18698_amd/build.py"
#endif

extern "C" {

const char *monarch_attn_last_error(void) { return g_err; }

const char *monarch_attn_build_id(void) { return MA_BUILD_ID; }

int monarch_attn_check(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    g_err[0] = '\0';
    return check_shape(N, d, m, b, T, dtype);
}

size_t monarch_attn_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b,
                                    int32_t T, int32_t dtype)
{
    if (B < 1 || H < 1 || check_shape(N, d, m, b, T, dtype) != MA_OK) return 0;
    return workspace_bytes(B * H, m * b, d, dtype);
}

int monarch_attn_release_workspace(void)
{
    g_err[0] = '\0';
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return fail(MA_EHIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> lock(g_dev_mutex);
    Device &D = g_dev[dev];
    bool synced = false;
    for (auto &entry : D.ws) {
        Workspace &w = *entry.second;
        std::lock_guard<std::mutex> wl(w.mu);
        if (!w.ptr && w.retired.empty()) continue;
        if (!synced) {
            if (hipDeviceSynchronize() != hipSuccess) return fail(MA_EHIP, "hipDeviceSynchronize failed");
            synced = true;
        }
        while (!w.retired.empty()) {
            if (hipFree(w.retired.back()) != hipSuccess) return fail(MA_EHIP, "freeing the workspace failed");
            w.retired.pop_back();
        }
        if (w.ptr && hipFree(w.ptr) != hipSuccess) return fail(MA_EHIP, "freeing the workspace failed");
        w.ptr = nullptr;
        w.bytes = 0;
        w.captured = false;
    }
    return MA_OK;
}

int monarch_attn_set_path(int32_t path)
{
    g_err[0] = '\0';
    if (path != kAuto && path != kHalfSteps && path != kFusedHead && path != kGrouped) {
        fail(MA_EINVAL, "unknown path %d", path);
        return -1;
    }
    return g_path.exchange(path);
}

int monarch_attn_timing_enable(int32_t flag)
{
    g_err[0] = '\0';
    std::lock_guard<std::mutex> lock(g_timing_mutex);
    if (flag && !g_timing.created) {
        for (int i = 0; i < 2 * kMaxLaunches; ++i) {
            if (hipEventCreate(&g_timing.ev[i]) != hipSuccess) return fail(MA_EHIP, "hipEventCreate failed");
        }
        g_timing.created = true;
    }
    g_timing.enabled = flag != 0;
    g_timing.ready = false;
    return MA_OK;
}

int32_t monarch_attn_timing_read(float *ms, int32_t *kind, int32_t cap)
{
    g_err[0] = '\0';
    std::lock_guard<std::mutex> lock(g_timing_mutex);
    if (!g_timing.ready) {
        fail(MA_EINVAL, "no timed call to read");
        return -1;
    }
    const int n = g_timing.nlaunch;
    if (hipEventSynchronize(g_timing.ev[2 * n - 1]) != hipSuccess) {
        fail(MA_EHIP, "hipEventSynchronize failed");
        return -1;
    }
    for (int i = 0; i < n && i < cap; ++i) {
        float t = 0.f;
        if (hipEventElapsedTime(&t, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]) != hipSuccess) {
            fail(MA_EHIP, "hipEventElapsedTime failed");
            return -1;
        }
        if (ms) ms[i] = t;
        if (kind) kind[i] = g_timing.kind[i];
    }
    return n;
}

int monarch_attn_fwd(const void *q, const void *k, const void *v, void *out, int64_t B, int64_t H, int64_t N,
                     int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream)
{
    return forward(q, k, v, out, nullptr, false, nullptr, false, B, H, N, d, m, b, T, dtype, stream);
}

int monarch_attn_fwd_noalloc(const void *q, const void *k, const void *v, void *out, int64_t B, int64_t H, int64_t N,
                             int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream)
{
    return forward(q, k, v, out, nullptr, false, nullptr, false, B, H, N, d, m, b, T, dtype, stream, true);
}

int monarch_attn_fwd_prepad(const void *q, const void *k, const void *v, void *out, const int32_t *lens, int64_t B,
                            int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype,
                            void *stream)
{
    return forward(q, k, v, out, nullptr, false, lens, lens != nullptr, B, H, N, d, m, b, T, dtype, stream, false, true);
}

int monarch_attn_fwd_varlen(const void *q, const void *k, const void *v, void *out, const int32_t *lens, int64_t B,
                            int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype,
                            void *stream)
{
    return forward(q, k, v, out, nullptr, false, lens, true, B, H, N, d, m, b, T, dtype, stream);
}

int monarch_attn_exact_fwd(const void *q, const void *k, const void *v, void *out, float *lse, int64_t B,
                           int64_t H, int64_t N, int64_t d, int32_t dtype, void *stream)
{
    g_err[0] = '\0';
    if (B < 0 || H < 0 || N < 0 || d < 1) return fail(MA_EINVAL, "B, H, N must be >= 0 and d >= 1");
    if (dtype != MA_F32 && dtype != MA_BF16 && dtype != MA_F16) return fail(MA_EINVAL, "unknown dtype %d", dtype);
    if (d > 128 || d % (16 / (int64_t)elem_bytes(dtype)) != 0)
        return fail(MA_EUNSUPPORTED, "d must be a multiple of %d up to 128 (got %lld)", (int)(16 / elem_bytes(dtype)),
                    (long long)d);
    if (B == 0 || H == 0 || N == 0) return MA_OK;  // nothing to compute: no launch, no pointer read
    if (!q || !k || !v || !out) return fail(MA_EINVAL, "null tensor pointer");
    if (N > 0x7fffffff) return fail(MA_EUNSUPPORTED, "N too large");
    int rc = check_heads(B, H, (N + 63) / 64);  // one workgroup per 64 query rows
    if (rc != MA_OK) return rc;
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)out) & 15u)
        return fail(MA_EINVAL, "q, k, v and out must be 16-byte aligned");
    if ((uintptr_t)lse & 3u) return fail(MA_EINVAL, "lse must be 4-byte aligned");
    const int64_t BH = B * H;
    const size_t tensor_bytes = (size_t)BH * N * d * elem_bytes(dtype);
    if (overlaps(out, tensor_bytes, q, tensor_bytes) || overlaps(out, tensor_bytes, k, tensor_bytes) ||
        overlaps(out, tensor_bytes, v, tensor_bytes))
        return fail(MA_EINVAL, "out must not overlap q, k or v");
    const size_t lse_bytes = (size_t)BH * N * sizeof(float);
    if (lse && (overlaps(lse, lse_bytes, q, tensor_bytes) || overlaps(lse, lse_bytes, k, tensor_bytes) ||
                overlaps(lse, lse_bytes, v, tensor_bytes) || overlaps(lse, lse_bytes, out, tensor_bytes)))
        return fail(MA_EINVAL, "lse must not overlap q, k, v or out");
    CallBufs bufs{q, k, v, out, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
    bool capturing = false;
    if ((rc = check_capture((hipStream_t)stream, capturing)) != MA_OK) return rc;
    std::unique_lock<std::mutex> tlock(g_timing_mutex);
    Launcher L{(hipStream_t)stream, g_timing.enabled};
    if (!L.timed) tlock.unlock();
    (void)hipGetLastError();
    switch (dtype) {
    case MA_F32: rc = run_exact<float>(L, bufs, lse, BH, (int)N, (int)d); break;
    case MA_BF16: rc = run_exact<__bf16>(L, bufs, lse, BH, (int)N, (int)d); break;
    default: rc = run_exact<_Float16>(L, bufs, lse, BH, (int)N, (int)d); break;
    }
    if (L.timed) {
        g_timing.nlaunch = L.n;
        g_timing.ready = (rc == MA_OK && L.n > 0);
    }
    if (rc != MA_OK) return rc;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(MA_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return MA_OK;
}

int monarch_attn_fwd_objective(const void *q, const void *k, const void *v, void *out, float *obj, int64_t B,
                               int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype,
                               void *stream)
{
    return forward(q, k, v, out, obj, true, nullptr, false, B, H, N, d, m, b, T, dtype, stream);
}

int monarch_attn_bwd(const void *q, const void *k, const void *v, const void *dout, void *dq, void *dk, void *dv,
                     int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype,
                     void *stream)
{
    return backward(q, k, v, dout, dq, dk, dv, nullptr, false, B, H, N, d, m, b, T, dtype, stream);
}

int monarch_attn_bwd_varlen(const void *q, const void *k, const void *v, const void *dout, void *dq, void *dk,
                            void *dv, const int32_t *lens, int64_t B, int64_t H, int64_t N, int64_t d, int64_t m,
                            int64_t b, int32_t T, int32_t dtype, void *stream)
{
    return backward(q, k, v, dout, dq, dk, dv, lens, true, B, H, N, d, m, b, T, dtype, stream);
}

int monarch_attn_bwd_check(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype)
{
    g_err[0] = '\0';
    return check_bwd_shape(N, d, m, b, T, dtype);
}

size_t monarch_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T,
                                        int32_t dtype)
{
    if (B < 1 || H < 1 || check_bwd_shape(N, d, m, b, T, dtype) != MA_OK) return 0;
    return bwd_layout(B * H, N, d, m, b, T, dtype).total();
}

}  // extern "C"

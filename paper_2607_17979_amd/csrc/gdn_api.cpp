// C ABI entry points: host-side argument checks, then the kernel launchers.
// No check touches the HIP runtime, so every error path can be exercised on a
// machine without a GPU.
#include "../../include/gdn.h"

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "gdn_device.h"
#include "gdn_launch.h"

static_assert(GDN_QK_L2NORM == gdn::kFlagQkL2Norm && GDN_GATE_LOGITS == gdn::kFlagGateLogits &&
                  GDN_SHORT_ONLY == gdn::kFlagShortOnly,
              "the ABI's flag bits are the kernels'");

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_heads(int H_qk, int H_v, int D_k, int D_v) {
    if (H_qk <= 0 || H_v <= 0)
        return fail(GDN_EINVAL, "head counts must be positive (H_qk=%d, H_v=%d)", H_qk, H_v);
    if (H_v % H_qk != 0)
        return fail(GDN_EINVAL, "H_v (%d) must be a multiple of H_qk (%d)", H_v, H_qk);
    if (D_k != D_v)
        return fail(GDN_EUNSUPPORTED, "d_k (%d) must equal d_v (%d)", D_k, D_v);
    if (D_k != 16 && D_k != 128)
        return fail(GDN_EUNSUPPORTED, "head dim %d unsupported (supported: 16, 128)", D_k);
    return GDN_OK;
}

int check_ptr16(const void* p, const char* name) {
    if (p == nullptr) return fail(GDN_EINVAL, "%s is NULL", name);
    if (!aligned(p, 16)) return fail(GDN_EALIGN, "%s is not 16-byte aligned", name);
    return GDN_OK;
}

int check_ptr4(const void* p, const char* name) {
    if (p == nullptr) return fail(GDN_EINVAL, "%s is NULL", name);
    if (!aligned(p, 4)) return fail(GDN_EALIGN, "%s is not 4-byte aligned", name);
    return GDN_OK;
}

int chunk_for(int D) { return D == 16 ? 16 : 64; }

}  // namespace

namespace gdn {

size_t prefill_workspace_bytes(int N) {
    if (N <= 0) return 0;
    return ((size_t)(N + 2) * sizeof(int32_t) + 255) / 256 * 256;
}

// Scratch of gdn_prefill_varlen_noalloc: the prefill workspace of up to
// kScratchMaxSeqs sequences in a file-scope device array, one copy per GPU,
// held until the process ends.  Host code uses it only through the device
// address hipGetSymbolAddress returns (the array's name on the host is a
// stand-in, not a device address).
constexpr int kScratchMaxSeqs = 16384;
constexpr size_t kScratchBytes = ((size_t)(kScratchMaxSeqs + 2) * sizeof(int32_t) + 255) / 256 * 256;
static __device__ __align__(256) int32_t scratch[kScratchBytes / sizeof(int32_t)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// The current device's address of `scratch`, looked up once per device with
// that device current.
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

}  // namespace gdn

extern "C" {

const char* gdn_last_error(void) { return g_last_error.c_str(); }

int gdn_abi_version(void) { return 210; }

static int decode_impl(const void* q, const void* k, const void* v, const float* g, const float* beta,
                       float* state, void* o, int B, int H_qk, int H_v, int D_k, int D_v, float scale,
                       int flags, void* stream) {
    if (B < 0) return fail(GDN_EINVAL, "B must be >= 0 (got %d)", B);
    if (int st = check_heads(H_qk, H_v, D_k, D_v)) return st;
    if (B == 0) return GDN_OK;
    if ((long long)B * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "B * H_v = %lld too large", (long long)B * H_v);
    int st;
    if ((st = check_ptr16(q, "q")) || (st = check_ptr16(k, "k")) || (st = check_ptr16(v, "v")) ||
        (st = check_ptr16(state, "state")) || (st = check_ptr16(o, "o")) ||
        (st = check_ptr4(g, "g")) || (st = check_ptr4(beta, "beta")))
        return st;
    gdn::DecodeArgs a{q, k, v, g, beta, state, o, B, H_qk, H_v, D_k, scale, nullptr, 0, flags};
    hipError_t e = gdn::launch_decode(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "decode launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

static int decode_indexed_impl(const void* q, const void* k, const void* v, const float* g,
                               const float* beta, float* state_pool, const int32_t* state_idx, void* o, int B,
                               int P, int H_qk, int H_v, int D_k, int D_v, float scale, int flags, void* stream) {
    if (B < 0) return fail(GDN_EINVAL, "B must be >= 0 (got %d)", B);
    if (P < 0) return fail(GDN_EINVAL, "P must be >= 0 (got %d)", P);
    if (int st = check_heads(H_qk, H_v, D_k, D_v)) return st;
    if (B == 0 || P == 0) return GDN_OK;
    if ((long long)B * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "B * H_v = %lld too large", (long long)B * H_v);
    if ((long long)P * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "P * H_v = %lld too large", (long long)P * H_v);
    int st;
    if ((st = check_ptr16(q, "q")) || (st = check_ptr16(k, "k")) || (st = check_ptr16(v, "v")) ||
        (st = check_ptr16(state_pool, "state_pool")) || (st = check_ptr4(state_idx, "state_idx")) ||
        (st = check_ptr16(o, "o")) || (st = check_ptr4(g, "g")) || (st = check_ptr4(beta, "beta")))
        return st;
    gdn::DecodeArgs a{q, k, v, g, beta, state_pool, o, B, H_qk, H_v, D_k, scale, state_idx, P, flags};
    hipError_t e = gdn::launch_decode(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "decode launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

size_t gdn_prefill_workspace_size(int N, int T, int H_v, int D_k, int D_v, int chunk) {
    if (N < 0 || T < 0 || H_v <= 0 || D_k != D_v || (D_k != 16 && D_k != 128) || chunk != chunk_for(D_k))
        return 0;
    return gdn::prefill_workspace_bytes(N);
}

}  // extern "C"

namespace {

// Checks of gdn_prefill_varlen's arguments other than the workspace; GDN_OK
// (with *noop set for N = 0) or the failing status with its message.
int check_prefill(const void* q, const void* k, const void* v, const float* g, const float* beta,
                  const int32_t* cu_seqlens, const float* initial_state, const float* final_state,
                  const void* o, int N, int T, int H_qk, int H_v, int D_k, int D_v, int chunk, bool* noop) {
    *noop = false;
    if (N < 0 || T < 0) return fail(GDN_EINVAL, "N and T must be >= 0 (N=%d, T=%d)", N, T);
    if (int st = check_heads(H_qk, H_v, D_k, D_v)) return st;
    if (chunk != chunk_for(D_k))
        return fail(GDN_EUNSUPPORTED, "chunk %d unsupported for head dim %d (use %d)", chunk, D_k,
                    chunk_for(D_k));
    if (N == 0) {
        *noop = true;
        return GDN_OK;
    }
    if ((long long)T * H_v > (1LL << 31) / 128 || (long long)N * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "problem too large (N=%d, T=%d, H_v=%d)", N, T, H_v);
    int st;
    if ((st = check_ptr4(cu_seqlens, "cu_seqlens")) || (st = check_ptr16(final_state, "final_state")))
        return st;
    if (initial_state != nullptr && !aligned(initial_state, 16))
        return fail(GDN_EALIGN, "initial_state is not 16-byte aligned");
    if (initial_state != nullptr && initial_state != final_state) {
        const char* a0 = reinterpret_cast<const char*>(initial_state);
        const char* b0 = reinterpret_cast<const char*>(final_state);
        const size_t bytes = (size_t)N * H_v * D_k * D_k * sizeof(float);
        if (a0 < b0 + bytes && b0 < a0 + bytes)
            return fail(GDN_EINVAL, "initial_state and final_state overlap without being equal");
    }
    if (T > 0) {
        if ((st = check_ptr16(q, "q")) || (st = check_ptr16(k, "k")) || (st = check_ptr16(v, "v")) ||
            (st = check_ptr16(o, "o")) || (st = check_ptr4(g, "g")) || (st = check_ptr4(beta, "beta")))
            return st;
    }
    return GDN_OK;
}

}  // namespace

extern "C" {

static int prefill_impl(const void* q, const void* k, const void* v, const float* g, const float* beta,
                        const int32_t* cu_seqlens, const float* initial_state, float* final_state, void* o,
                        int N, int T, int H_qk, int H_v, int D_k, int D_v, int chunk, float scale, int flags,
                        void* workspace, size_t workspace_bytes, void* stream) {
    bool noop;
    if (int st = check_prefill(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o, N, T, H_qk, H_v,
                               D_k, D_v, chunk, &noop))
        return st;
    if (noop) return GDN_OK;
    const size_t need = gdn::prefill_workspace_bytes(N);
    if (workspace == nullptr || workspace_bytes < need)
        return fail(GDN_EWORKSPACE, "workspace of %zu bytes needed, %zu given%s", need,
                    workspace_bytes, workspace == nullptr ? " (NULL)" : "");
    if (!aligned(workspace, 256)) return fail(GDN_EALIGN, "workspace is not 256-byte aligned");
    gdn::PrefillArgs a{q, k, v, g, beta, cu_seqlens, initial_state, final_state, o,
                       N, T, H_qk, H_v, D_k, chunk, scale, workspace, nullptr, 0, false, flags};
    hipError_t e = gdn::launch_prefill(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "prefill launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

int gdn_prefill_varlen_noalloc(const void* q, const void* k, const void* v, const float* g,
                               const float* beta, const int32_t* cu_seqlens, const float* initial_state,
                               float* final_state, void* o, int N, int T, int H_qk, int H_v, int D_k,
                               int D_v, int chunk, float scale, void* stream) {
    g_last_error.clear();
    bool noop;
    if (int st = check_prefill(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o, N, T, H_qk, H_v,
                               D_k, D_v, chunk, &noop))
        return st;
    if (noop) return GDN_OK;
    if (N > gdn::kScratchMaxSeqs)
        return fail(GDN_EWORKSPACE, "N = %d sequences exceeds the %d the no-allocation entry point's "
                    "static scratch holds (use gdn_prefill_varlen with a workspace)", N, gdn::kScratchMaxSeqs);
    void* ws = nullptr;
    hipError_t e = gdn::scratch_address(&ws);
    if (e != hipSuccess) return fail(GDN_EHIP, "scratch lookup failed: %s", hipGetErrorString(e));
    gdn::PrefillArgs a{q, k, v, g, beta, cu_seqlens, initial_state, final_state, o,
                       N, T, H_qk, H_v, D_k, chunk, scale, ws, nullptr, 0, false, 0};
    e = gdn::launch_prefill(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "prefill launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

static int prefill_indexed_impl(const void* q, const void* k, const void* v, const float* g,
                                const float* beta, const int32_t* cu_seqlens, float* state_pool,
                                const int32_t* state_idx, void* o, int N, int T, int P, int H_qk, int H_v,
                                int D_k, int D_v, int chunk, float scale, int flags, void* workspace,
                                size_t workspace_bytes, void* stream) {
    if (N < 0 || T < 0) return fail(GDN_EINVAL, "N and T must be >= 0 (N=%d, T=%d)", N, T);
    if (P < 0) return fail(GDN_EINVAL, "P must be >= 0 (got %d)", P);
    if (int st = check_heads(H_qk, H_v, D_k, D_v)) return st;
    if (chunk != chunk_for(D_k))
        return fail(GDN_EUNSUPPORTED, "chunk %d unsupported for head dim %d (use %d)", chunk, D_k,
                    chunk_for(D_k));
    if (N == 0 || P == 0) return GDN_OK;
    if ((long long)T * H_v > (1LL << 31) / 128 || (long long)N * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "problem too large (N=%d, T=%d, H_v=%d)", N, T, H_v);
    if ((long long)P * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "P * H_v = %lld too large", (long long)P * H_v);
    int st;
    if ((st = check_ptr4(cu_seqlens, "cu_seqlens")) || (st = check_ptr16(state_pool, "state_pool")) ||
        (st = check_ptr4(state_idx, "state_idx")))
        return st;
    if (T > 0) {
        if ((st = check_ptr16(q, "q")) || (st = check_ptr16(k, "k")) || (st = check_ptr16(v, "v")) ||
            (st = check_ptr16(o, "o")) || (st = check_ptr4(g, "g")) || (st = check_ptr4(beta, "beta")))
            return st;
    }
    const size_t need = gdn::prefill_workspace_bytes(N);
    if (workspace == nullptr || workspace_bytes < need)
        return fail(GDN_EWORKSPACE, "workspace of %zu bytes needed, %zu given%s", need,
                    workspace_bytes, workspace == nullptr ? " (NULL)" : "");
    if (!aligned(workspace, 256)) return fail(GDN_EALIGN, "workspace is not 256-byte aligned");
    gdn::PrefillArgs a{q, k, v, g, beta, cu_seqlens, state_pool, state_pool, o,
                       N, T, H_qk, H_v, D_k, chunk, scale, workspace, state_idx, P, false, flags};
    hipError_t e = gdn::launch_prefill(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "prefill launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

static int multitoken_impl(const void* q, const void* k, const void* v, const float* g, const float* beta,
                           const int32_t* cu_seqlens, float* state, const int32_t* state_idx, int P, void* o,
                           int N, int T, int H_qk, int H_v, int D_k, int D_v, float scale, int flags,
                           void* workspace, size_t workspace_bytes, void* stream) {
    if (N < 0 || T < 0) return fail(GDN_EINVAL, "N and T must be >= 0 (N=%d, T=%d)", N, T);
    if (int st = check_heads(H_qk, H_v, D_k, D_v)) return st;
    if (D_k != 128) return fail(GDN_EUNSUPPORTED, "multi-token decode runs for head dim 128 (got %d)", D_k);
    if ((long long)T > (long long)gdn::kRecurMax * N)
        return fail(GDN_EINVAL, "T = %d > %d N: some sequence has more than %d tokens", T, gdn::kRecurMax,
                    gdn::kRecurMax);
    if (N == 0) return GDN_OK;
    if ((long long)N * H_v > (1LL << 30))
        return fail(GDN_EINVAL, "problem too large (N=%d, H_v=%d)", N, H_v);
    int st;
    if ((st = check_ptr4(cu_seqlens, "cu_seqlens")) || (st = check_ptr16(state, "state"))) return st;
    if (state_idx != nullptr) {
        if (P < 0) return fail(GDN_EINVAL, "P must be >= 0 (got %d)", P);
        if (P == 0) return GDN_OK;
        if ((long long)P * H_v > (1LL << 30)) return fail(GDN_EINVAL, "P * H_v = %lld too large", (long long)P * H_v);
        if ((st = check_ptr4(state_idx, "state_idx"))) return st;
    }
    if (T > 0) {
        if ((st = check_ptr16(q, "q")) || (st = check_ptr16(k, "k")) || (st = check_ptr16(v, "v")) ||
            (st = check_ptr16(o, "o")) || (st = check_ptr4(g, "g")) || (st = check_ptr4(beta, "beta")))
            return st;
    }
    const size_t need = gdn::prefill_workspace_bytes(N);
    if (workspace == nullptr || workspace_bytes < need)
        return fail(GDN_EWORKSPACE, "workspace of %zu bytes needed, %zu given%s", need,
                    workspace_bytes, workspace == nullptr ? " (NULL)" : "");
    if (!aligned(workspace, 256)) return fail(GDN_EALIGN, "workspace is not 256-byte aligned");
    gdn::PrefillArgs a{q, k, v, g, beta, cu_seqlens, state, state, o,
                       N, T, H_qk, H_v, D_k, chunk_for(D_k), scale, workspace, state_idx, P, true, flags};
    hipError_t e = gdn::launch_prefill(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(GDN_EHIP, "multi-token decode launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

int gdn_decode(const void* q, const void* k, const void* v, const float* g, const float* beta,
               float* state, void* o, int B, int H_qk, int H_v, int D_k, int D_v, float scale,
               void* stream) {
    g_last_error.clear();
    return decode_impl(q, k, v, g, beta, state, o, B, H_qk, H_v, D_k, D_v, scale, 0, stream);
}

int gdn_decode_indexed(const void* q, const void* k, const void* v, const float* g, const float* beta,
                       float* state_pool, const int32_t* state_idx, void* o, int B, int P, int H_qk,
                       int H_v, int D_k, int D_v, float scale, void* stream) {
    g_last_error.clear();
    return decode_indexed_impl(q, k, v, g, beta, state_pool, state_idx, o, B, P, H_qk, H_v, D_k, D_v, scale, 0,
                               stream);
}

int gdn_prefill_varlen(const void* q, const void* k, const void* v, const float* g,
                       const float* beta, const int32_t* cu_seqlens, const float* initial_state,
                       float* final_state, void* o, int N, int T, int H_qk, int H_v, int D_k,
                       int D_v, int chunk, float scale, void* workspace, size_t workspace_bytes,
                       void* stream) {
    g_last_error.clear();
    return prefill_impl(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o, N, T, H_qk, H_v, D_k, D_v,
                        chunk, scale, 0, workspace, workspace_bytes, stream);
}

int gdn_prefill_varlen_indexed(const void* q, const void* k, const void* v, const float* g,
                               const float* beta, const int32_t* cu_seqlens, float* state_pool,
                               const int32_t* state_idx, void* o, int N, int T, int P, int H_qk,
                               int H_v, int D_k, int D_v, int chunk, float scale, void* workspace,
                               size_t workspace_bytes, void* stream) {
    g_last_error.clear();
    return prefill_indexed_impl(q, k, v, g, beta, cu_seqlens, state_pool, state_idx, o, N, T, P, H_qk, H_v, D_k,
                                D_v, chunk, scale, 0, workspace, workspace_bytes, stream);
}

int gdn_decode_multitoken(const void* q, const void* k, const void* v, const float* g,
                          const float* beta, const int32_t* cu_seqlens, float* state, void* o, int N,
                          int T, int H_qk, int H_v, int D_k, int D_v, float scale, void* workspace,
                          size_t workspace_bytes, void* stream) {
    g_last_error.clear();
    return multitoken_impl(q, k, v, g, beta, cu_seqlens, state, nullptr, 0, o, N, T, H_qk, H_v, D_k, D_v, scale,
                           0, workspace, workspace_bytes, stream);
}

int gdn_decode_ex(const void* q, const void* k, const void* v, const float* g, const float* beta,
                  float* state, const int32_t* state_idx, int P, void* o, int B, int H_qk, int H_v, int D_k,
                  int D_v, float scale, int flags, void* stream) {
    g_last_error.clear();
    if (flags & ~(GDN_QK_L2NORM | GDN_GATE_LOGITS))
        return fail(GDN_EINVAL, "unknown or unsupported flags 0x%x for gdn_decode_ex", flags);
    if (state_idx == nullptr)
        return decode_impl(q, k, v, g, beta, state, o, B, H_qk, H_v, D_k, D_v, scale, flags, stream);
    return decode_indexed_impl(q, k, v, g, beta, state, state_idx, o, B, P, H_qk, H_v, D_k, D_v, scale, flags,
                               stream);
}

int gdn_prefill_varlen_ex(const void* q, const void* k, const void* v, const float* g, const float* beta,
                          const int32_t* cu_seqlens, const float* initial_state, float* final_state,
                          const int32_t* state_idx, int P, void* o, int N, int T, int H_qk, int H_v, int D_k,
                          int D_v, int chunk, float scale, int flags, void* workspace, size_t workspace_bytes,
                          void* stream) {
    g_last_error.clear();
    if (flags & ~(GDN_QK_L2NORM | GDN_GATE_LOGITS | GDN_SHORT_ONLY))
        return fail(GDN_EINVAL, "unknown flags 0x%x for gdn_prefill_varlen_ex", flags);
    const int prologue = flags & (GDN_QK_L2NORM | GDN_GATE_LOGITS);
    if ((state_idx != nullptr || (flags & GDN_SHORT_ONLY)) && initial_state != nullptr &&
        initial_state != final_state)
        return fail(GDN_EINVAL, "with state_idx or GDN_SHORT_ONLY the state is updated in place: "
                    "initial_state must be NULL or equal final_state");
    if (flags & GDN_SHORT_ONLY) {
        if (D_k == 128 && D_v == 128 && chunk != 64)
            return fail(GDN_EUNSUPPORTED, "chunk %d unsupported for head dim 128 (use 64)", chunk);
        return multitoken_impl(q, k, v, g, beta, cu_seqlens, final_state, state_idx, P, o, N, T, H_qk, H_v, D_k,
                               D_v, scale, prologue, workspace, workspace_bytes, stream);
    }
    if (state_idx != nullptr)
        return prefill_indexed_impl(q, k, v, g, beta, cu_seqlens, final_state, state_idx, o, N, T, P, H_qk, H_v,
                                    D_k, D_v, chunk, scale, prologue, workspace, workspace_bytes, stream);
    return prefill_impl(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o, N, T, H_qk, H_v, D_k, D_v,
                        chunk, scale, prologue, workspace, workspace_bytes, stream);
}

}  // extern "C"

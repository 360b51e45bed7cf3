// C ABI of the binary-delta matmul library: argument checks, path choice and
// kernel launches.  Everything here runs on the host.  The only allocation is
// the grouped prefill's partial-sum workspace, made once per (device, stream)
// on first need and kept until the process ends.
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "../../include/bitdelta.h"
#include "internal.h"

// The allocation-free entry point's scratch (see device_scratch below).
constexpr size_t kScratchBytes = bitdelta::kPrefillSplitBytes;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kSkinnyRows = 64;
// Batched requests with at least this many rows take the grouped fused GEMM
// (one pass over W per output tile) rather than the decode-shaped kernel,
// which streams W once per 64 rows.
constexpr int kGroupedMinRows = 256;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int elem_size(int dtype) {
    switch (dtype) {
        case BITDELTA_F32: return 4;
        case BITDELTA_BF16: return 2;
        case BITDELTA_F16: return 2;
        case BITDELTA_I8: return 1;
        default: return 0;
    }
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
    if (a == nullptr || b == nullptr || abytes == 0 || bbytes == 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

int hip_status(hipError_t e) { return e == hipSuccess ? BITDELTA_OK : BITDELTA_ERR_HIP; }

// The launchers report hipGetLastError() after their launches; an error left
// behind by an earlier, unrelated runtime call of the caller (a not-ready
// query, say) would otherwise be reported as this call's launch failure.
void clear_stale_error() { (void)hipGetLastError(); }

// Largest extent any kernel indexes with 32-bit arithmetic.
constexpr int64_t kMaxDim = (int64_t)1 << 30;

int check_matmul(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w, int64_t N,
                 const uint32_t* packed, const float* alpha, const int32_t* tenant_ids,
                 int32_t T, int in_dtype, void* y, int y_dtype) {
    if (M < 0 || N < 0 || K < 0 || T < 1) return BITDELTA_ERR_SHAPE;
    if (K % 32 != 0) return BITDELTA_ERR_SHAPE;
    if (M > kMaxDim || N > kMaxDim || K > kMaxDim) return BITDELTA_ERR_SHAPE;
    if (in_dtype != BITDELTA_BF16 && in_dtype != BITDELTA_F16) return BITDELTA_ERR_DTYPE;
    if (y_dtype != BITDELTA_F32 && y_dtype != in_dtype) return BITDELTA_ERR_DTYPE;
    if (M == 0 || N == 0) return BITDELTA_OK;
    if (y == nullptr || alpha == nullptr) return BITDELTA_ERR_NULL;
    if (K > 0 && (x == nullptr || w == nullptr || packed == nullptr)) return BITDELTA_ERR_NULL;
    if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y, 16)) return BITDELTA_ERR_ALIGN;
    if (!aligned(packed, 4) || !aligned(alpha, 4) || !aligned(tenant_ids, 4)) return BITDELTA_ERR_ALIGN;
    const size_t ybytes = (size_t)M * (size_t)N * (size_t)elem_size(y_dtype);
    if (overlaps(y, ybytes, x, (size_t)M * K * 2) || overlaps(y, ybytes, w, (size_t)N * K * 2) ||
        overlaps(y, ybytes, packed, (size_t)T * N * (K / 32) * 4) ||
        overlaps(y, ybytes, alpha, (size_t)T * 4) ||
        overlaps(y, ybytes, tenant_ids, tenant_ids ? (size_t)M * 4 : 0))
        return BITDELTA_ERR_ALIAS;
    return BITDELTA_OK;
}

// Validation mode (BITDELTA_VALIDATE set and not "0"): read the tenant ids back
// through a fixed host buffer, in chunks, and report any id outside [0, T).
bool validation_mode() {
    const char* v = getenv("BITDELTA_VALIDATE");
    return v != nullptr && v[0] != '\0' && strcmp(v, "0") != 0;
}

int check_tenant_ids(const int32_t* ids, int64_t M, int32_t T, hipStream_t stream) {
    constexpr int64_t kChunk = 1024;
    int32_t buf[kChunk];
    for (int64_t off = 0; off < M; off += kChunk) {
        const int64_t n = M - off < kChunk ? M - off : kChunk;
        if (hipMemcpyAsync(buf, ids + off, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
                hipSuccess ||
            hipStreamSynchronize(stream) != hipSuccess)
            return BITDELTA_ERR_HIP;
        for (int64_t i = 0; i < n; ++i)
            if (buf[i] < 0 || buf[i] >= T) return BITDELTA_ERR_TENANT;
    }
    return BITDELTA_OK;
}

// Partial-sum workspace of the grouped prefill split, one per (device,
// stream): two calls on one stream run in order, so they can share it, while
// calls on different streams may overlap and must not.  Allocated on first
// need (never while the stream is being captured into a graph: such a call
// runs without the split) and kept until the process ends.  Every call writes
// what it reads there, so the contents need no initial value.
// Allocation failure or a full table also mean "no split", never an error.
struct Workspace {
    int device;
    hipStream_t stream;
    void* ptr;
};
constexpr int kMaxWorkspaces = 64;
std::mutex g_ws_mutex;
Workspace g_ws[kMaxWorkspaces];
int g_ws_count = 0;

void* stream_workspace(hipStream_t stream, size_t bytes) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    for (int i = 0; i < g_ws_count; ++i)
        if (g_ws[i].device == dev && g_ws[i].stream == stream) return g_ws[i].ptr;
    if (g_ws_count == kMaxWorkspaces) return nullptr;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return nullptr;
    g_ws[g_ws_count++] = {dev, stream, p};
    return p;
}

// Scratch of the allocation-free entry point: one fixed device array, each
// GPU holding its own copy for the life of the process.  Host code reaches it
// only through the address hipGetSymbolAddress gives for the current device
// (the array's name is not a device address on the host); that address is
// taken once per device, on the device's first allocation-free call.  Its
// size is the grouped prefill's full split, so the allocation-free calls split
// exactly as bitdelta_matmul does.  Every call writes what it reads there:
// nothing has to start at zero.  Calls that overlap on one GPU share it and
// race.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, or null if the runtime cannot
// give it.
void* device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

// More output tiles than CUs is possible (the grouped GEMM may split).
bool grouped_may_split(int64_t M, int64_t N, int32_t T) {
    const int64_t U = T < M ? T : M;
    const int64_t tiles_m = (M + 255 * U) / 256, tiles_n = (N + 255) / 256;
    return tiles_m * tiles_n > 256;
}

int choose_path(int64_t M, int64_t N, int64_t K, int32_t T, int has_tenant_ids) {
    if (M <= kSkinnyRows) return BITDELTA_PATH_SKINNY;
    if (!has_tenant_ids) return BITDELTA_PATH_PREFILL;
    if (M >= kGroupedMinRows && M <= kMaxDim && N <= kMaxDim && K <= kMaxDim &&
        bitdelta::prefill_grouped_supported((int)M, (int)N, (int)K, T))
        return BITDELTA_PATH_PREFILL;
    return BITDELTA_PATH_SKINNY;
}

}  // namespace

extern "C" {

int bitdelta_version(void) { return 100; }

const char* bitdelta_status_string(int status) {
    switch (status) {
        case BITDELTA_OK: return "ok";
        case BITDELTA_ERR_NULL: return "a required pointer is NULL";
        case BITDELTA_ERR_SHAPE: return "invalid shape (negative size, K not a multiple of 32, T < 1 or size too large)";
        case BITDELTA_ERR_ALIGN: return "pointer not aligned as required";
        case BITDELTA_ERR_DTYPE: return "dtype not accepted for this argument";
        case BITDELTA_ERR_UNSUPPORTED: return "request not supported by the selected path";
        case BITDELTA_ERR_HIP: return "HIP runtime error at launch";
        case BITDELTA_ERR_ALIAS: return "output overlaps an input";
        case BITDELTA_ERR_TENANT: return "a tenant id is outside [0, T) (validation mode)";
        default: return "unknown status";
    }
}

int bitdelta_pack(const void* signs, int in_dtype, int64_t rows, int64_t K, uint32_t* packed,
                  hipStream_t stream) {
    const int es = elem_size(in_dtype);
    if (es == 0) return BITDELTA_ERR_DTYPE;
    if (rows < 0 || K < 0 || K % 32 != 0) return BITDELTA_ERR_SHAPE;
    if (rows == 0 || K == 0) return BITDELTA_OK;
    if (signs == nullptr || packed == nullptr) return BITDELTA_ERR_NULL;
    if (!aligned(signs, 4 * es) || !aligned(packed, 4)) return BITDELTA_ERR_ALIGN;
    if (overlaps(packed, (size_t)rows * (K / 32) * 4, signs, (size_t)rows * K * es))
        return BITDELTA_ERR_ALIAS;
    // the sign bit of both 16-bit formats is bit 15: one kernel serves both
    if (in_dtype == BITDELTA_F16) in_dtype = BITDELTA_BF16;
    clear_stale_error();
    return hip_status(bitdelta::launch_pack(signs, in_dtype, rows * K, packed, stream));
}

int bitdelta_unpack(const uint32_t* packed, int64_t rows, int64_t K, void* signs, int out_dtype,
                    hipStream_t stream) {
    const int es = elem_size(out_dtype);
    if (es == 0) return BITDELTA_ERR_DTYPE;
    if (rows < 0 || K < 0 || K % 32 != 0) return BITDELTA_ERR_SHAPE;
    if (rows == 0 || K == 0) return BITDELTA_OK;
    if (signs == nullptr || packed == nullptr) return BITDELTA_ERR_NULL;
    if (!aligned(signs, 4 * es) || !aligned(packed, 4)) return BITDELTA_ERR_ALIGN;
    if (overlaps(packed, (size_t)rows * (K / 32) * 4, signs, (size_t)rows * K * es))
        return BITDELTA_ERR_ALIAS;
    clear_stale_error();
    return hip_status(bitdelta::launch_unpack(packed, rows * K, signs, out_dtype, stream));
}

int bitdelta_compress(const uint16_t* w_fine, const uint16_t* w_base, int64_t rows, int64_t K,
                      int in_dtype, uint32_t* packed, float* row_abs_sum, float* alpha,
                      hipStream_t stream) {
    if (in_dtype != BITDELTA_BF16 && in_dtype != BITDELTA_F16) return BITDELTA_ERR_DTYPE;
    if (rows < 0 || K < 0 || K % 32 != 0 || rows > kMaxDim || K > kMaxDim) return BITDELTA_ERR_SHAPE;
    if (rows == 0 || K == 0) return BITDELTA_OK;
    if (w_fine == nullptr || w_base == nullptr || packed == nullptr || row_abs_sum == nullptr)
        return BITDELTA_ERR_NULL;
    if (!aligned(w_fine, 16) || !aligned(w_base, 16) || !aligned(packed, 4) ||
        !aligned(row_abs_sum, 4) || !aligned(alpha, 4))
        return BITDELTA_ERR_ALIGN;
    const size_t wbytes = (size_t)rows * K * 2, pbytes = (size_t)rows * (K / 32) * 4,
                 rbytes = (size_t)rows * 4, abytes = alpha ? 4 : 0;
    if (overlaps(packed, pbytes, w_fine, wbytes) || overlaps(packed, pbytes, w_base, wbytes) ||
        overlaps(row_abs_sum, rbytes, w_fine, wbytes) || overlaps(row_abs_sum, rbytes, w_base, wbytes) ||
        overlaps(row_abs_sum, rbytes, packed, pbytes) || overlaps(alpha, abytes, w_fine, wbytes) ||
        overlaps(alpha, abytes, w_base, wbytes) || overlaps(alpha, abytes, packed, pbytes) ||
        overlaps(alpha, abytes, row_abs_sum, rbytes))
        return BITDELTA_ERR_ALIAS;
    clear_stale_error();
    return hip_status(bitdelta::launch_compress(w_fine, w_base, (int)rows, (int)K, in_dtype, packed,
                                                row_abs_sum, alpha, stream));
}

int bitdelta_matmul_path(int64_t M, int64_t N, int64_t K, int32_t T, int has_tenant_ids) {
    return choose_path(M, N, K, T, has_tenant_ids);
}

}  // extern "C"

namespace {

// The matmul behind every entry point.  noalloc: the grouped prefill's
// partial sums go to the static scratch array instead of the per-stream
// workspace, and nothing is allocated.
int matmul_impl(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w_base, int64_t N,
                const uint32_t* packed_s, const float* alpha, const int32_t* tenant_ids, int32_t T,
                int in_dtype, void* y, int y_dtype, int path, hipStream_t stream, bool noalloc) {
    int rc = check_matmul(x, M, K, w_base, N, packed_s, alpha, tenant_ids, T, in_dtype, y, y_dtype);
    if (rc != BITDELTA_OK) return rc;
    if (path == BITDELTA_PATH_AUTO) path = choose_path(M, N, K, T, tenant_ids != nullptr);
    if (path != BITDELTA_PATH_SKINNY && path != BITDELTA_PATH_PREFILL) return BITDELTA_ERR_UNSUPPORTED;
    if (path == BITDELTA_PATH_PREFILL && tenant_ids != nullptr &&
        !bitdelta::prefill_grouped_supported((int)M, (int)N, (int)K, T))
        return BITDELTA_ERR_UNSUPPORTED;
    if (M == 0 || N == 0) return BITDELTA_OK;
    if (tenant_ids != nullptr && validation_mode()) {
        rc = check_tenant_ids(tenant_ids, M, T, stream);
        if (rc != BITDELTA_OK) return rc;
    }
    const int et = in_dtype;
    clear_stale_error();

    if (path == BITDELTA_PATH_PREFILL && tenant_ids != nullptr) {
        void* ws = nullptr;
        size_t ws_bytes = 0;
        if (grouped_may_split(M, N, T)) {
            if (noalloc) {
                ws = device_scratch();
                if (ws == nullptr) return BITDELTA_ERR_HIP;
                ws_bytes = kScratchBytes;
            } else {
                ws_bytes = bitdelta::prefill_split_bytes();
                ws = stream_workspace(stream, ws_bytes);
                (void)hipGetLastError();  // a failed allocation only disables the split
            }
        }
        return hip_status(bitdelta::launch_prefill_grouped(x, (int)M, (int)K, w_base, (int)N,
                                                           packed_s, alpha, tenant_ids, (int)T, y,
                                                           y_dtype, et, stream, ws, ws ? ws_bytes : 0));
    }
    if (path == BITDELTA_PATH_PREFILL)
        return hip_status(bitdelta::launch_prefill(x, (int)M, (int)K, w_base, (int)N, packed_s,
                                                   alpha, y, y_dtype, et, stream));

    // Skinny path: 64 rows per launch (each launch streams W once more).
    const int es = elem_size(y_dtype);
    for (int64_t r0 = 0; r0 < M; r0 += kSkinnyRows) {
        const int rows = (int)(M - r0 < kSkinnyRows ? M - r0 : kSkinnyRows);
        rc = hip_status(bitdelta::launch_skinny(
            x + r0 * K, rows, (int)K, w_base, (int)N, packed_s, alpha,
            tenant_ids ? tenant_ids + r0 : nullptr, (int)T,
            static_cast<char*>(y) + r0 * N * es, y_dtype, et, stream));
        if (rc != BITDELTA_OK) return rc;
    }
    return BITDELTA_OK;
}

}  // namespace

extern "C" {

int bitdelta_matmul_typed(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w_base,
                          int64_t N, const uint32_t* packed_s, const float* alpha,
                          const int32_t* tenant_ids, int32_t T, int in_dtype, void* y,
                          int y_dtype, int path, hipStream_t stream) {
    return matmul_impl(x, M, K, w_base, N, packed_s, alpha, tenant_ids, T, in_dtype, y, y_dtype, path,
                       stream, false);
}

int bitdelta_matmul_noalloc(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w_base,
                            int64_t N, const uint32_t* packed_s, const float* alpha,
                            const int32_t* tenant_ids, int32_t T, int in_dtype, void* y,
                            int y_dtype, int path, hipStream_t stream) {
    return matmul_impl(x, M, K, w_base, N, packed_s, alpha, tenant_ids, T, in_dtype, y, y_dtype, path,
                       stream, true);
}

int bitdelta_matmul_with_path(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w_base,
                              int64_t N, const uint32_t* packed_s, const float* alpha,
                              const int32_t* tenant_ids, int32_t T, void* y, int y_dtype,
                              int path, hipStream_t stream) {
    return bitdelta_matmul_typed(x, M, K, w_base, N, packed_s, alpha, tenant_ids, T, BITDELTA_BF16,
                                 y, y_dtype, path, stream);
}

int bitdelta_matmul(const uint16_t* x, int64_t M, int64_t K, const uint16_t* w_base, int64_t N,
                    const uint32_t* packed_s, const float* alpha, const int32_t* tenant_ids,
                    int32_t T, void* y, int y_dtype, hipStream_t stream) {
    return bitdelta_matmul_typed(x, M, K, w_base, N, packed_s, alpha, tenant_ids, T, BITDELTA_BF16,
                                 y, y_dtype, BITDELTA_PATH_AUTO, stream);
}

}  // extern "C"

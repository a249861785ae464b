// spccl_compress_static: compression for callers that cannot allocate.
//
// It runs the one-launch compression kernels (each 16384-element partition
// finds its offset from its predecessors' counts, so the only scratch is a
// status word, one look-back word per partition and one per 256 partitions)
// with that scratch in a file-scope device array instead of a caller
// workspace.  Every GPU the library runs on holds
// its own copy of the array, at its own address, until the process ends.  In
// host code the array's name is not a device address, so the address of each
// device's copy is taken once (hipGetSymbolAddress, with that device current)
// and only that address reaches kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "spccl_internal.h"
#include "../../include/spccl.h"

namespace spccl {
spccl_status_t launch_to_pici_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, hipStream_t st);
spccl_status_t launch_fill_zero(void* p, uint64_t bytes, hipStream_t st);
}  // namespace spccl

using namespace spccl;

namespace {

constexpr uint64_t kStaticMaxParts = SPCCL_STATIC_MAX_ELEMS / kPartElems;
static_assert(SPCCL_STATIC_MAX_ELEMS % kPartElems == 0, "the maximum is a whole number of partitions");
// a look-back word per partition and one per kPlaceChunk partitions (the chunk sums)
constexpr uint64_t kStaticFlagWords = kStaticMaxParts + (kStaticMaxParts + kPlaceChunk - 1) / kPlaceChunk;
constexpr uint64_t kStaticScratchBytes = kWsFlagsOffset + 8 * kStaticFlagWords;

static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];           // each device's copy of `scratch`, once looked up

// The device address of the current device's copy of the array.
spccl_status_t scratch_ptr(uint8_t** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SPCCL_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SPCCL_ERR_HIP;
        g_ptr[dev] = p;
    }
    *out = static_cast<uint8_t*>(g_ptr[dev]);
    return SPCCL_OK;
}

// Look-back words carry a per-launch epoch, so the array never needs clearing
// between calls; these epochs are drawn only for this array.
std::atomic<uint32_t> g_epoch{1};

// A device-side wait that ran past its spin limit leaves a status in the
// control block; the message then may not hold the right offsets, so its
// magic is cleared and every reader rejects it as corrupt.
__global__ void k_static_check(const WsCtrl* ctrl, uint8_t* out) {
    if (threadIdx.x == 0 && ctrl->status != 0u) *reinterpret_cast<uint32_t*>(out) = 0u;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline uint64_t elem(int32_t dt) { return dt == kBF16 ? 2 : 4; }

}  // namespace

extern "C" spccl_status_t spccl_compress_static(const void* dense, uint64_t n, int32_t dtype, void* out,
                                                uint64_t out_bytes, void* stream) {
    if (dtype != kF32 && dtype != kBF16) return SPCCL_ERR_UNSUPPORTED;
    if (n > SPCCL_STATIC_MAX_ELEMS) return SPCCL_ERR_UNSUPPORTED;
    if ((n && (!dense || (reinterpret_cast<uintptr_t>(dense) & (elem(dtype) - 1)))) || !out || !aligned16(out))
        return SPCCL_ERR_INVALID_ARG;
    if (out_bytes < spccl_stream_bound(n, dtype)) return SPCCL_ERR_CAPACITY;
    const uintptr_t d = reinterpret_cast<uintptr_t>(dense), o = reinterpret_cast<uintptr_t>(out);
    if (n && d < o + out_bytes && o < d + n * elem(dtype)) return SPCCL_ERR_INVALID_ARG;
    uint8_t* ws = nullptr;
    spccl_status_t st = scratch_ptr(&ws);
    if (st != SPCCL_OK) return st;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    // the sticky status must start clear: a fill kernel, not a memset node
    if ((st = launch_fill_zero(ws, sizeof(uint32_t), hs)) != SPCCL_OK) return st;
    PiciSinkArgs g{};
    g.slots = nullptr;                       // single pass: no value slots
    g.a = DevOperand{nullptr, static_cast<const uint8_t*>(dense), n * elem(dtype)};
    g.out = static_cast<uint8_t*>(out);
    g.n = n;
    g.T = num_tiles(n);
    g.nparts = (uint32_t)num_parts(n);
    g.epoch = g_epoch.fetch_add(1, std::memory_order_relaxed) & 0x3FFFFFFFu;
    g.ctrl = reinterpret_cast<WsCtrl*>(ws);
    g.flags = reinterpret_cast<uint64_t*>(ws + kWsFlagsOffset);
    if ((st = launch_to_pici_dt(dtype, SRC_DENSE, SRC_NONE, g, hs)) != SPCCL_OK) return st;
    hipLaunchKernelGGL(k_static_check, dim3(1), dim3(64), 0, hs, reinterpret_cast<const WsCtrl*>(ws),
                       static_cast<uint8_t*>(out));
    return hipGetLastError() == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
}

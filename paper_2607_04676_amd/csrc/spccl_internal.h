// Internal constants and layout helpers of the gfx950 Pici library.  Host and
// device code of the library share this header; nothing outside the library
// includes it.
#pragma once
#include <stdint.h>

namespace spccl {

constexpr uint32_t kMagic = 0x49434950u;        // "PICI"
constexpr uint64_t kHeaderBytes = 48;
constexpr uint64_t kNnzUnknown = ~0ull;
constexpr uint32_t kTileElems = 4096;           // a 64 x 64 virtual tile
constexpr uint32_t kWave = 64;                  // CDNA wavefront
constexpr uint32_t kWavesPerBlock = 4;          // one tile per wave
constexpr uint32_t kBlockThreads = kWave * kWavesPerBlock;
constexpr uint32_t kTilesPerPart = kWavesPerBlock;   // look-back partition = one block
constexpr uint32_t kStageBytes = 7168;          // LDS staging per wave (an fp32 tile up to 7/16 full in one go)

constexpr int kFmtDense = 0, kFmtPici = 1, kFmtCoo = 2;
constexpr int kKindArray = 0, kKindStream = 1;
constexpr int kF32 = 0, kBF16 = 1;

// Workspace: a control block, then one 64-bit look-back word per partition.
struct WsCtrl {
    uint32_t status;     // sticky device status (first error wins)
    uint32_t pad[63];
};
static_assert(sizeof(WsCtrl) == 256, "control block is 256 bytes");
constexpr uint64_t kWsFlagsOffset = sizeof(WsCtrl);

__host__ __device__ inline uint64_t elem_bytes(int dtype) { return dtype == kBF16 ? 2 : 4; }
__host__ __device__ inline uint64_t num_tiles(uint64_t n) { return (n + kTileElems - 1) / kTileElems; }
__host__ __device__ inline uint64_t off_I(uint64_t n) { return kHeaderBytes + 512ull * num_tiles(n); }
__host__ __device__ inline uint64_t off_A(uint64_t n) {
    return (off_I(n) + 4ull * (num_tiles(n) + 1) + 15ull) & ~15ull;
}
__host__ __device__ inline uint64_t pici_bytes(uint64_t n, int dtype, uint64_t nnz) {
    return off_A(n) + nnz * elem_bytes(dtype);
}
__host__ __device__ inline uint64_t dense_msg_bytes(uint64_t n, int dtype) {
    return kHeaderBytes + n * elem_bytes(dtype);
}
// COO message: header, J (nnz 32-bit flat indices, increasing) at 48, zero
// pad to 16 bytes, V (nnz values) at coo_off_V(nnz).
__host__ __device__ inline uint64_t coo_off_V(uint64_t nnz) { return (kHeaderBytes + 4ull * nnz + 15ull) & ~15ull; }
__host__ __device__ inline uint64_t coo_bytes(int dtype, uint64_t nnz) {
    return coo_off_V(nnz) + nnz * elem_bytes(dtype);
}
constexpr uint64_t kPartElems = (uint64_t)kTilesPerPart * kTileElems;

__host__ __device__ inline uint64_t num_parts(uint64_t n) {
    uint64_t T = num_tiles(n);
    uint64_t p = (T + kTilesPerPart - 1) / kTilesPerPart;
    return p ? p : 1;
}

// The second pass of a two-pass Pici sink sums the partitions' aggregates per
// chunk of kPlaceChunk partitions; each chunk's sum has a look-back word of its
// own, after the partitions' words.
constexpr uint32_t kPlaceChunk = 256;
__host__ __device__ inline uint64_t num_place_chunks(uint64_t nparts) {
    return (nparts + kPlaceChunk - 1) / kPlaceChunk;
}
// look-back words of a workspace for n elements: one per partition, one per chunk
__host__ __device__ inline uint64_t flag_words(uint64_t n) {
    const uint64_t p = num_parts(n);
    return p + num_place_chunks(p);
}

// A fresh 30-bit epoch for the look-back words of one launch (host).
uint32_t next_epoch();

// Source kinds of the tile pipeline.
enum SrcKind { SRC_NONE = 0, SRC_DENSE = 1, SRC_PICI = 2, SRC_COO = 3 };

// A reduce / codec operand as the kernels see it.
struct DevOperand {
    const uint8_t* hdr;    // message header, or nullptr for a raw array
    const uint8_t* data;   // raw array base, or the message base for Pici / COO
    uint64_t cap;          // capacity of the message buffer in bytes
    const uint64_t* idx;   // COO: idx[t] = epoch << 32 | first entry of tile t (T + 1 words, k_coo_index),
                           // or nullptr: search J
    uint32_t idx_epoch;    // the epoch of this call's index words; a tile whose words carry another searches J
};

struct PiciSinkArgs {
    DevOperand a, b;
    uint8_t* out;          // output message base
    uint64_t n;
    uint64_t T;
    uint32_t nparts;
    uint32_t epoch;        // tags this call's look-back words (unique per launch)
    WsCtrl* ctrl;
    uint64_t* flags;
    uint8_t* slots;        // two-pass mode: one worst-case slot of compacted values per partition
    uint32_t* idx_slots;   // COO output: one worst-case slot of flat indices per partition
};

struct DenseSinkArgs {
    DevOperand a, b;
    uint8_t* out_hdr;      // nullptr for an ARRAY output
    uint8_t* out;          // output element base
    uint64_t n;
    uint64_t T;
    WsCtrl* ctrl;
};

constexpr int kMaxGatherParts = 64;
struct GatherArgs {
    DevOperand part[kMaxGatherParts];
    uint8_t* out;          // element base of part 0 of this launch
    uint64_t n;            // elements per part
    uint64_t T;
    WsCtrl* ctrl;
};

// Sliced streams: slot q of a stream holds elements [kSliceElems q, ...) as
// an ordinary message; one block (4 tiles) produces or consumes one slice.
constexpr uint64_t kSliceElems = kPartElems;
__host__ __device__ inline uint64_t num_slices(uint64_t n) { return (n + kSliceElems - 1) / kSliceElems; }
__host__ __device__ inline uint64_t slice_slot_bytes(int dtype) {
    const uint64_t p = pici_bytes(kSliceElems, dtype, kSliceElems), d = dense_msg_bytes(kSliceElems, dtype);
    return p > d ? p : d;
}

enum SlicedOp { kSlicedCompress = 0, kSlicedReduceToSliced = 1, kSlicedReduceToDense = 2, kSlicedExpand = 3 };

struct SlicedArgs {
    const uint8_t* a;      // dense input array, or a sliced stream (expand, copy)
    const uint8_t* b;      // sliced input stream, or nullptr
    uint8_t* out;          // sliced output stream, or dense output array
    uint64_t n;            // elements
    uint64_t slot;         // bytes per slot
    double thresh;         // a produced slice is dense iff its sparsity <= thresh (tracked: iff the
                           // tracker's estimate <= thresh)
    WsCtrl* ctrl;
    double* track;         // per slice: sigma0, sigma_prev (nullptr: decide on the measured sparsity)
    int32_t track_step;    // 0: the first send (sigma0 := measured); 1: a later one (Eq. 7 estimate)
    uint8_t* fmt_out;      // per slice: the format produced (nullptr: not recorded)
};

// One sliced ring step for up to kMaxBatchRanks virtual ranks in a single
// launch (grid y = rank): rank r's arguments are base with its own dense or
// source pointer a[r], its own dense output (out_dense[r], else the strided
// stream base.out + r out_stride), its threshold, and strided received
// streams, trackers and format records.
constexpr int kMaxBatchRanks = 32;
struct SlicedBatch {
    SlicedArgs base;
    const uint8_t* a[kMaxBatchRanks];
    uint8_t* out_dense[kMaxBatchRanks];
    double thresh[kMaxBatchRanks];
    uint64_t b_stride, out_stride;   // bytes between ranks
    uint64_t track_stride;           // doubles between ranks
    uint64_t fmt_stride;             // bytes between ranks
};

// One step of the canonical ring for a batch of virtual ranks in a single
// launch (grid y = the rank's place in the batch): each rank's operands,
// output, look-back words and value slots; sizes, the epoch, capacities and
// the status word are the launch's base arguments, shared.  An operand
// pointer replaces the base operand's (a message keeps its header-to-data
// offset); a null b leaves the base's b.
// Per rank of a ring whose formats are decided on the device: its sigma0 and
// tracked sparsity (Sec. IV-C), and the formats of the message it receives
// and of the one it sends at the current step.
struct RingRank {
    double sigma0, sigma_prev;
    int32_t in_fmt, out_fmt;
};

struct RankBatch {
    const uint8_t* a[kMaxBatchRanks];
    const uint8_t* b[kMaxBatchRanks];
    uint8_t* out[kMaxBatchRanks];
    uint8_t* flags[kMaxBatchRanks];     // the rank's look-back words (zeroed once per collective)
    uint8_t* slots[kMaxBatchRanks];     // the rank's value slots (two-pass Pici sink)
    // With gate set, a rank takes part only if its decided formats match
    // gate_in / gate_out (-1: any); rank[j] indexes gate for batch entry j.
    const RingRank* gate;
    int32_t gate_in, gate_out;
    int32_t rank[kMaxBatchRanks];
};

// The decisions of one canonical ring step on the device (k_ring_decide):
// rank r's last send is the message at slots0 + r * slot_bytes.
enum RingDecide {
    kDecideFirst = 0,     // after the first compression: sigma0, the first send's format
    kDecideStep = 1,      // before ring step `step`: the previous step's trace, this step's formats
    kDecideGather = 2,    // all-reduce transition, before encoding: the gather's formats
    kDecideGatherSizes = 3,  // after the transition's encoding: its sizes in the trace
    kDecideAllGather = 4  // a standalone all-gather's sends (every part Pici): their trace
};

struct RingArgs {
    RingRank* rr;             // P entries
    void* trace;              // spccl_trace_t[P * (P - 1) + P] in device memory
    const uint8_t* slots0;
    uint64_t slot_bytes;
    uint64_t m;               // elements per message
    int32_t P, step, mode, dtype;
    double intra, inter, ag;  // the policy's thresholds
    int32_t ranks_per_node, adaptive;
};

__host__ __device__ inline bool rank_skipped(const RankBatch& rb, uint32_t j) {
    if (!rb.gate) return false;
    const RingRank& q = rb.gate[rb.rank[j]];
    return (rb.gate_in >= 0 && q.in_fmt != rb.gate_in) || (rb.gate_out >= 0 && q.out_fmt != rb.gate_out);
}

__host__ __device__ inline DevOperand rebase(DevOperand o, const uint8_t* p) {
    if (o.hdr) {
        o.data = p + (o.data - o.hdr);
        o.hdr = p;
    } else {
        o.data = p;
    }
    return o;
}

__host__ __device__ inline PiciSinkArgs rank_sink(PiciSinkArgs g, const RankBatch& rb, uint32_t r) {
    g.a = rebase(g.a, rb.a[r]);
    if (rb.b[r]) g.b = rebase(g.b, rb.b[r]);
    g.out = rb.out[r];
    g.flags = reinterpret_cast<uint64_t*>(rb.flags[r]);
    g.slots = rb.slots[r];
    return g;
}

__host__ __device__ inline DenseSinkArgs rank_dense(DenseSinkArgs g, const RankBatch& rb, uint32_t r) {
    g.a = rebase(g.a, rb.a[r]);
    if (rb.b[r]) g.b = rebase(g.b, rb.b[r]);
    if (g.out_hdr) {
        g.out_hdr = rb.out[r];
        g.out = rb.out[r] + kHeaderBytes;
    } else {
        g.out = rb.out[r];
    }
    return g;
}

__host__ __device__ inline SlicedArgs batch_rank(const SlicedBatch& b, uint32_t r) {
    SlicedArgs g = b.base;
    g.a = b.a[r];
    if (g.b) g.b = b.base.b + r * b.b_stride;
    g.out = b.out_dense[r] ? b.out_dense[r] : b.base.out + r * b.out_stride;
    g.thresh = b.thresh[r];
    if (g.track) g.track = b.base.track + r * b.track_stride;
    if (g.fmt_out) g.fmt_out = b.base.fmt_out + r * b.fmt_stride;
    return g;
}

}  // namespace spccl

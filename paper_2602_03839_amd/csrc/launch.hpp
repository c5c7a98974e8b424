// launch.hpp -- kernel parameter blocks and launcher declarations shared by
// the kernels and the C ABI layer.  Parameter blocks travel as kernel
// arguments (they stay below the 4 KiB kernel-argument limit), so a batched
// call needs no device-side descriptor table and no extra copy.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

constexpr int kMaxBatch = 64;  // tensors per launch; larger batches are split
static_assert(kMaxBatch <= 64, "the tile -> tensor lookup keeps one tensor per lane");

// Tile shapes: compute threads per block (a multiple of 64; one more wave is
// added for the scan) and 8-element groups per thread.  The defaults give
// 16-wave blocks (15 compute + 1 scan), one per CU: waves are handed out to
// the SIMDs in fours, and the sparsifier's LDS value ring takes 150 KiB of the
// CU's 160 KiB.
// Refresh writes of a tensor whose inference copy mirrors its snapshot cover
// whole aligned runs of kSectorLanes x 8 elements (16 bytes per lane).
// 8 lanes = one 128-byte cache line: a scattered write costs about the same
// HBM time whatever its size up to a line, so whole lines need the fewest
// write requests (at ~1% density 45% of the lines change, against one request
// per change for 2-byte writes).
constexpr int kEncodeTB = 960;
constexpr int kEncodeU = 2;
constexpr int kSectorLanes = 8;
constexpr int kLocoTB = 960;

struct EncodeTensorDesc {
  const float* w_new;
  const uint16_t* snap;
  uint16_t* refresh;
  uint64_t n;
  uint32_t index_base;
  uint32_t mirror;  // refresh holds snap's bits on entry: whole-sector refresh writes
};

struct EncodeParams {
  uint64_t* ws;
  uint32_t* idx;
  uint16_t* val;
  uint64_t capacity;
  uint64_t* count;
  uint64_t* seg_begin;  // already offset to this launch's first tensor; may be null
  uint32_t ntiles;
  int ntensors;
  uint32_t tile_begin[kMaxBatch + 1];
  EncodeTensorDesc t[kMaxBatch];
};

// Receivers that compute in a lower precision than BF16 (App. D).
constexpr int kDtypeFp8 = 1;    // OCP FP8 E4M3, per-tensor FP32 scale
constexpr int kDtypeMxfp4 = 2;  // OCP MXFP4: E8M0 scale per 32 values, E2M1 codes

struct LocoTensorDesc {
  const float* delta;
  float* residual;
  const float* theta;
  uint64_t n;
  uint32_t index_base;
  float inv_scale;  // FP8 gate: the receiver's per-tensor scale
};

struct LocoParams {
  uint64_t* ws;
  uint32_t* idx;
  float* val;
  uint64_t capacity;
  uint64_t* count;
  uint64_t* seg_begin;
  float tau;
  int gate_dtype;  // with theta: 0 = BF16 gate, kDtypeFp8 / kDtypeMxfp4 = that receiver's gate
  int gm;          // kernel form, the same for every launch of a call (sets the tile size):
                  // 0 = threshold, 1 = BF16 gate, 2 = FP8 gate, 3 = MXFP4 gate
  uint32_t ntiles;
  int ntensors;
  uint32_t tile_begin[kMaxBatch + 1];
  LocoTensorDesc t[kMaxBatch];
};

struct ApplyTensorDesc {
  uint16_t* dst;
  uint64_t n;
  uint32_t index_base;
};

struct ApplyParams {
  const uint32_t* idx;
  const uint16_t* val;
  uint64_t capacity;
  const uint64_t* seg_begin;  // device [ntensors] (batched form), or the single `begin`
  const uint64_t* end;
  uint64_t* rejected;
  int ntensors;
  ApplyTensorDesc t[kMaxBatch];
};

constexpr int kMaxLists = 8;  // workers' lists per outer-step launch

struct OuterTensorDesc {
  float* theta;
  float* momentum;
  uint64_t n;
  uint32_t index_base;
};

struct OuterListDesc {
  const uint32_t* idx;
  const float* val;
  uint64_t capacity;
  const uint64_t* seg_begin;  // device [ntensors], offset to this launch's first tensor
  const uint64_t* end;        // device: end of this launch's last tensor's entries
};

struct OuterParams {
  uint32_t nunits;
  int ntensors;
  int nlists;
  float mu;
  float alpha;
  uint32_t tile_begin[kMaxBatch + 1];  // first work unit of each tensor
  OuterTensorDesc t[kMaxBatch];
  OuterListDesc l[kMaxLists];
};

struct VarintEncParams {
  uint64_t* ws;
  const uint32_t* idx;
  uint64_t capacity;           // entries readable in idx
  const uint64_t* end;         // device: entries in the list
  const uint64_t* seg_begin;   // device [nseg], may be null (one segment)
  uint32_t nseg;
  uint8_t* out;
  uint64_t out_capacity;
  uint64_t* seg_bytes;         // device [nseg], may be null
  uint64_t* total;             // device
};

struct VarintDecParams {
  uint64_t* ws;
  const uint8_t* in;
  uint64_t in_capacity;
  const uint64_t* nbytes;      // device: bytes in the stream
  const uint64_t* seg_begin;   // device [nseg], may be null (one segment)
  uint32_t nseg;
  uint32_t* idx;
  uint64_t capacity;           // entries writable in idx
  uint64_t* count;             // device: entries decoded
};

// Receivers that compute in a lower precision D (App. D); kDtypeFp8 and
// kDtypeMxfp4 are defined above LocoParams.

struct LowpTensorDesc {
  const float* w_new;
  const uint8_t* snap;         // FP8: n codes; MXFP4: (n + 1) / 2 bytes of packed codes
  const uint8_t* snap_scales;  // MXFP4: (n + 31) / 32 scale bytes
  uint64_t n;
  uint32_t index_base;
  float inv_scale;             // FP8: the receiver computes with fl32(w * inv_scale)
};

struct LowpParams {
  uint64_t* ws;
  uint32_t* idx;
  void* val;  // FP8: uint8 codes; MXFP4: uint16 (scale << 8) | code
  uint64_t capacity;
  uint64_t* count;
  uint64_t* seg_begin;
  uint32_t ntiles;
  int ntensors;
  uint32_t tile_begin[kMaxBatch + 1];
  LowpTensorDesc t[kMaxBatch];
};

struct LowpApplyTensorDesc {
  uint8_t* codes;
  uint8_t* scales;  // MXFP4 only
  uint64_t n;
  uint32_t index_base;
};

struct LowpApplyParams {
  const uint32_t* idx;
  const void* val;
  uint64_t capacity;
  const uint64_t* seg_begin;
  const uint64_t* end;
  uint64_t* rejected;
  int ntensors;
  int dtype;
  LowpApplyTensorDesc t[kMaxBatch];
};

static_assert(sizeof(LowpParams) < 4096, "kernel argument block too large");
static_assert(sizeof(LowpApplyParams) < 4096, "kernel argument block too large");

// Weight hash: a tree of SHA-256 over 16 KiB chunks ("leaves") of the
// concatenated BF16 bytes.  The tensors' pointers and stream offsets go to a
// device table in the caller's workspace, written by small setup launches
// that also gather the leaves which do not lie inside one tensor (a boundary
// between tensors falls inside them) into one 16 KiB scratch slot each.
constexpr uint64_t kHashLeafElems = 8192;
constexpr uint64_t kHashLeafBytes = 2 * kHashLeafElems;
constexpr int kHashSetupBatch = 64;
constexpr uint32_t kHashTreeFan = 512;  // digests reduced by one tree block

struct HashEntry {
  const uint16_t* ptr;
  uint64_t off;  // stream offset (elements) of the tensor's first value
};

struct HashCopyJob {
  const uint16_t* src;
  uint64_t dst;    // byte offset in the scratch slots
  uint64_t count;  // values
};

struct HashSetupParams {
  HashEntry* table;
  uint8_t* scratch;
  uint32_t first_entry;
  uint32_t nentries;
  uint32_t njobs;
  HashEntry entries[kHashSetupBatch];
  HashCopyJob jobs[kHashSetupBatch];
};

struct HashLeafParams {
  const HashEntry* table;  // ntensors entries + one whose off is the stream length
  uint32_t ntensors;
  const uint8_t* scratch;  // slot t: the leaf that starts inside tensor t, if gathered
  uint8_t* digests;        // out: nleaves x 32 bytes
  uint64_t nleaves;
  uint64_t total;          // stream length in values
};

// A leaf [x, x + le) that starts inside the tensor [off, end) is read in place
// when it ends inside that tensor and its last aligned 4-byte word does too
// (the kernel reads whole words; the tensor's base is 4-byte aligned).
__host__ __device__ inline bool hash_leaf_in_place(uint64_t x, uint64_t le, uint64_t off,
                                                   uint64_t end) {
  const uint64_t lend = x + le;
  return lend <= end && (((lend - off) & 1) == 0 || lend < end);
}

static_assert(sizeof(HashSetupParams) < 4096, "kernel argument block too large");
struct CooEncParams {
  uint64_t* ws;
  const uint32_t* idx;
  uint64_t capacity;
  const uint64_t* end;         // device: entries in the patch
  const uint64_t* seg_begin;   // device [nseg]
  uint32_t nseg;
  const uint32_t* cols;        // device [nseg]: columns of each tensor
  uint32_t* first;             // device [nseg]: each segment's first index
  uint8_t* drow;
  uint16_t* dcol;
  uint64_t out_capacity;       // pairs writable
  uint64_t* seg_pairs;         // device [nseg]: where each segment's pairs start
  uint64_t* total;             // device: pairs in the stream
};

struct CooDecParams {
  uint64_t* ws;
  const uint8_t* drow;
  const uint16_t* dcol;
  uint64_t pair_capacity;      // pairs readable
  const uint64_t* npairs;      // device: pairs in the stream
  const uint64_t* seg_begin;   // device [nseg]: entry where each segment starts
  const uint64_t* seg_pairs;   // device [nseg]: pair where each segment starts
  uint32_t nseg;
  const uint32_t* cols;        // device [nseg]
  const uint32_t* first;       // device [nseg]
  const uint64_t* nent;        // device: entries in the patch
  uint32_t* idx;
  uint64_t capacity;
};

static_assert(sizeof(EncodeParams) < 4096, "kernel argument block too large");
static_assert(sizeof(OuterParams) < 4096, "kernel argument block too large");
static_assert(sizeof(LocoParams) < 4096, "kernel argument block too large");
static_assert(sizeof(ApplyParams) < 4096, "kernel argument block too large");

uint32_t encode_tile_elems();
uint32_t loco_tile_elems(int gm);
hipError_t launch_encode(EncodeParams& p, hipStream_t stream);
hipError_t launch_loco(LocoParams& p, hipStream_t stream);

// Two-pass form of the threshold sparsifier (loco2.hip): tiles of kL2Tile
// elements, each staging up to kL2Cap selected entries; the ordering passes
// work on units of kL2Unit tiles.  Its staging area (loco2_scratch_bytes for
// a launch of ntiles tiles) lies in the caller's workspace past the fixed
// part.  p.ntiles counts kL2Tile-element tiles.
constexpr uint32_t kL2Tile = 1024;
constexpr uint32_t kL2Cap = 128;
constexpr uint32_t kL2Unit = 256;
size_t loco2_scratch_bytes(uint32_t ntiles);
hipError_t launch_loco2(LocoParams& p, void* scratch, hipStream_t stream);
hipError_t launch_apply(const ApplyParams& p, hipStream_t stream);
hipError_t launch_cast(const float* src, uint16_t* dst, uint64_t n, hipStream_t stream);
// p[0 .. nwords) = 0 by a kernel (not a memset, so a captured graph replays it as a kernel)
hipError_t launch_zero_words(uint64_t* p, uint64_t nwords, hipStream_t stream);
uint64_t outer_unit_elems();
// Largest capacity (entries, bytes or pairs) the index-stream kernels take.
uint64_t stream_max_items();
hipError_t launch_varint_encode(const VarintEncParams& p, hipStream_t stream);
hipError_t launch_varint_decode(const VarintDecParams& p, hipStream_t stream);
hipError_t launch_coo_encode(const CooEncParams& p, hipStream_t stream);
hipError_t launch_coo_decode(const CooDecParams& p, hipStream_t stream);
hipError_t launch_outer(const OuterParams& p, hipStream_t stream);
uint32_t lowp_tile_elems();
hipError_t launch_encode_lowp(int dtype, LowpParams& p, hipStream_t stream);
hipError_t launch_apply_lowp(const LowpApplyParams& p, hipStream_t stream);
hipError_t launch_cast_lowp(int dtype, const float* src, uint64_t n, float inv_scale,
                            uint8_t* codes, uint8_t* scales, hipStream_t stream);
hipError_t launch_hash_setup(const HashSetupParams& p, hipStream_t stream);
hipError_t launch_hash_leaves(const HashLeafParams& p, hipStream_t stream);
hipError_t launch_hash_tree(const uint8_t* in, uint64_t n_in, uint8_t* out, hipStream_t stream);

}  // namespace pulse

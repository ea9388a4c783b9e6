// Internal tables and kernel launchers of the LayerCheck HIP library.
// Shared by the host runtime (lc_runtime.cpp) and the kernels (lc_kernels.hip,
// lc_optim.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lc {

// ---- tiling ------------------------------------------------------------------
// Score: a chunk is a run of consecutive elements of one segment holding
// kChunkBytes of weights (and the same of shadow).  Chunks never cross a
// segment, so every layer owns a contiguous range of chunks and one fp64
// (sum|W-S|, sum|S|) pair per chunk is reduced in a fixed order per layer.
#ifndef LC_CHUNK_BYTES
#define LC_CHUNK_BYTES (8u * 1024u)
#endif
#ifndef LC_XCD_REMAP
#define LC_XCD_REMAP 1
#endif
#ifndef LC_XCD_RUN
#define LC_XCD_RUN 0  // 0: each XCD takes one contiguous eighth; g > 0: interleaved runs of g items
#endif
#ifndef LC_MAX_GRID_BLOCKS
#define LC_MAX_GRID_BLOCKS 0  // 0: only the dispatch limit caps a grid (testing builds set it low)
#endif
#ifndef LC_PIECE_BYTES
#define LC_PIECE_BYTES (8u * 1024u)
#endif
constexpr uint32_t kScoreThreads = 256;
constexpr uint32_t kChunkBytes = LC_CHUNK_BYTES;
// Pack/restore: a piece is kPieceBytes of one copy unit (one array of one
// segment); records are laid out so that every unit starts 256-B aligned.
constexpr uint32_t kCopyThreads = 256;
constexpr uint32_t kPieceBytes = LC_PIECE_BYTES;
static_assert(kChunkBytes % (16u * kScoreThreads) == 0, "score tiling: whole vectors per thread");
static_assert(kPieceBytes % (16u * kCopyThreads) == 0, "pack tiling");
constexpr uint32_t kRecordAlign = 256u;
constexpr uint32_t kFinalizeThreads = 1024;
constexpr uint32_t kSelectThreads = 256;

// Resident blocks per CU of the streaming kernels (0: as many as registers
// and waves allow), held there by a dynamic LDS reservation the kernel never
// touches.  Fewer streams open at once let HBM turn between reads and writes
// less often; kernels that only read, and kernels that end each block with a
// reduction (its tail leaves the block's slot without loads in flight), want
// more.  Measured on
// MI355X, same arrays, one process (GB/s, unreserved -> reserved):
//   ACCUM score (two reads, one write), 4 per CU: 8B 6425 -> 6688,
//     70B shard 6230 -> 6324, 13B 6070 -> 6158, Qwen2.5-14B 6414 -> 6574;
//     2 per CU loses 14%, 3 ties 4 on the larger states;
//   SNAPSHOT score (two reads), 5 per CU: 8B 6960 -> 7224, 13B 7069 -> 7232,
//     Qwen2.5-14B 6590 -> 6733, 70B shard 6990 -> 7219 (3 and 4 per CU lose);
//   pack and unpack (copies), 6 per CU: +0.2..1.8% (3 per CU: -12%);
//   fused AdamW, 2 per CU: 5930 -> 6004; fused SGD: no gain at 2..6.
#ifndef LC_SCORE_ACCUM_BLOCKS_PER_CU
#define LC_SCORE_ACCUM_BLOCKS_PER_CU 4
#endif
#ifndef LC_SCORE_SNAPSHOT_BLOCKS_PER_CU
#define LC_SCORE_SNAPSHOT_BLOCKS_PER_CU 5
#endif
#ifndef LC_COPY_BLOCKS_PER_CU
#define LC_COPY_BLOCKS_PER_CU 6
#endif
#ifndef LC_ADAMW_BLOCKS_PER_CU
#define LC_ADAMW_BLOCKS_PER_CU 2
#endif
#ifndef LC_SGD_BLOCKS_PER_CU
#define LC_SGD_BLOCKS_PER_CU 0
#endif
// Dynamic LDS bytes per block that leave room for at most `blocks_per_cu`
// blocks on a CU of the current device (0 when blocks_per_cu is 0 or the
// device's limits leave no such size).
uint32_t occupancy_lds(uint32_t blocks_per_cu);

// One segment as the score kernel sees it.
struct ScoreSeg {
  uint64_t w;            // device address of the weights
  uint64_t s;            // device address of the shadow
  uint64_t numel;
  uint32_t chunk_begin;  // global index of the segment's first chunk
  uint32_t vec_ok;       // w and s both 16-B aligned
};

// One block of a layer record: one array (W, master, m or v) of one segment.
struct CopyUnit {
  uint64_t arr;      // device address of the array range
  uint64_t shadow;   // shadow range for W units, 0 otherwise
  uint64_t rec_off;  // byte offset of the block inside the record (256-B aligned)
  uint64_t bytes;    // payload bytes (the block is padded to kRecordAlign)
  uint32_t piece0;   // first layer-local piece index of this unit
  uint32_t vec_ok;   // arr (and shadow) 16-B aligned
  uint32_t elem;     // element size in bytes (2 or 4)
  uint32_t pad;
};

// One segment as the optimizer kernels see it (static part).
struct OptSeg {
  uint64_t w;            // weights (bf16 or fp32)
  uint64_t master;       // fp32 master, 0 when absent
  uint64_t m;            // fp32 Adam first moment (AdamW only)
  uint64_t v;            // fp32 Adam second moment (AdamW only)
  uint64_t numel;
  uint32_t chunk_begin;  // same chunks as the score kernel
  uint32_t vec_ok;       // master/m/v 16-B aligned and weights aligned to 4 elements
};

// Per-call part: gradient address and weight-decay flag of each segment.
struct GradSeg {
  uint64_t grad;
  uint32_t decay;
  uint32_t vec_ok;  // gradient aligned to 4 elements
};

// fp32 scalars of one AdamW step, formed in fp64 on the host and rounded once.
struct AdamScalars {
  float b1, omb1, b2, omb2, c1, c2, eps, lr, decay;
};

// fp32 scalars of one SGD step: lr and the decoupled decay factor 1 - lr wd.
struct SgdScalars {
  float lr, decay;
};

// Written by the select kernel to device memory and to a pinned host mirror,
// followed by the 0/1 mask of n_layers bytes.  In the mirror `seq` is written
// last, after a system-scope fence: the host waits for the number it passed
// to the kernel instead of synchronising the stream.
struct SelectHeader {
  uint32_t n_selected;
  uint32_t n_forced;
  uint64_t payload_bytes;
  int64_t max_age;
  double weighted_age;
  uint64_t total_pieces;
  uint64_t age_numerator;
  uint64_t seq;
  uint64_t reserved;
};
static_assert(sizeof(SelectHeader) == 64, "header layout");

// Device-resident state of one context.
struct DeviceTables {
  uint32_t n_layers;
  uint32_t n_chunks;
  int dtype;  // 1 bf16, 2 f32
  int mode;   // 0 accum, 1 snapshot
  double eps_w;
  int64_t s_max;

  const ScoreSeg* segs;
  const uint32_t* chunk_seg;          // [n_chunks]
  const uint32_t* layer_chunk_begin;  // [N+1]
  double2* partials;                  // [n_chunks] (sum|W-S|, sum|S|)
  double* u;                          // [N]
  double* delta;                      // [N]
  int64_t* t_last;                    // [N]
  const double* k0;                   // [N]
  const uint64_t* numel;              // [N]
  const uint64_t* rec_bytes;          // [N]
  const uint64_t* layer_pieces;       // [N] pieces of one record
  const CopyUnit* units;              // all units, layer-major, record order
  const uint32_t* piece_unit;         // layout-wide piece -> unit index
  const uint64_t* layer_piece_begin;  // [N+1] offset of each layer in piece_unit
  uint32_t* sel_layer;                // [N] layer of each selected rank
  uint64_t* sel_rec_prefix;           // [N+1] record byte offsets by rank
  uint64_t* sel_piece_prefix;         // [N+1] piece offsets by rank
  SelectHeader* result;               // header + mask[N]
  SelectHeader* host_result;          // pinned host mirror of result (device address)
  const OptSeg* opt_segs;             // [n_segments]
  const GradSeg* grad_segs;           // [n_segments], refreshed per optimizer call
  // restore scratch
  uint32_t* rank_layer;               // [N]
  uint64_t* rank_src;                 // [N]
  uint64_t* rank_piece_prefix;        // [N+1]
};

// Launchers: return hipGetLastError() of the launches.
// launch_score: score kernel, then the finalize kernel (u and Delta).
hipError_t launch_score(const DeviceTables& t, hipStream_t st);
// Eq. 1-2 from the per-chunk partials alone (after an optimizer step).
hipError_t launch_finalize(const DeviceTables& t, hipStream_t st);
hipError_t launch_select(const DeviceTables& t, int64_t step, double lr_scale, int base_mode, uint64_t seq,
                         hipStream_t st);
hipError_t launch_pack(const DeviceTables& t, uint32_t first_rank, uint32_t last_rank,
                       uint64_t piece_base, uint64_t n_pieces, uint64_t rec_base,
                       void* staging, int refresh_shadow, hipStream_t st);
hipError_t launch_unpack(const DeviceTables& t, uint32_t n_ranks, uint64_t n_pieces,
                         hipStream_t st);
// Optimizer steps writing the per-chunk drift partials (lc_optim.hip).
hipError_t launch_adamw(const DeviceTables& t, int grad_dtype, int has_master, const AdamScalars& sc,
                        hipStream_t st);
hipError_t launch_sgd(const DeviceTables& t, int grad_dtype, int has_master, const SgdScalars& sc, hipStream_t st);

}  // namespace lc

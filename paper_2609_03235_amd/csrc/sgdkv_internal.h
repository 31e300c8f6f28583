// Internal interface between the C-ABI host layer (sgdkv_host.cpp) and the
// HIP kernels. Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sgdkv {

constexpr int kMaxKvHeads = 64;    // per-head tables travel by value in kernel arguments
constexpr int kMaxSplitRows = 512; // window rows one score workgroup holds (a row split)
constexpr int kMaxGroupRows = 4096; // G*w rows of one KV head's window queries, over all row splits
constexpr int kMaxDecodeGroup = 16;
constexpr int kMaxCompactSegs = 512;  // decode segments whose workgroup table travels in the kernel arguments
constexpr int kMaxIptQHeads = 256;  // query heads per layer the Ipt. aggregations accept
constexpr int kBlock = 256;        // threads per workgroup in every kernel but the decode split
#ifndef SGDKV_DECODE_BLOCK
#define SGDKV_DECODE_BLOCK 256
#endif
constexpr int kDecodeBlock = SGDKV_DECODE_BLOCK;  // threads per decode-split workgroup: one split per wave
constexpr int kDecodeWaves = kDecodeBlock / 64;   // splits a decode workgroup merges into one partial
constexpr int kLseTile = 128;      // keys staged in LDS per step of score pass 1
constexpr int kColTileBf16 = 128;  // keys staged in LDS per step of score pass 2 (bf16 keys)
constexpr int kColTileF32 = 64;    // the same for fp32 keys (LDS holds half as many)
constexpr int kScoreChunkQuantum = 128;  // score chunks are whole tiles of both passes
constexpr int kScoreWorkgroups = 256;   // workgroups that fill the MI355X (its compute units): score launches aim at it
constexpr int kHistChunkMax = 8192;      // positions per pooling / radix-pass workgroup, at most
constexpr int kPoolHalo = 64;            // pooling radii up to this are staged in LDS
constexpr int kChunkHistWords = 260;     // a scored chunk's last-digit histogram and count above (16-byte rows)
constexpr int kCopyRows = 64;            // output rows per work item of the row gather
#ifndef SGDKV_SCORE_WAVES
#define SGDKV_SCORE_WAVES 8
#endif
constexpr int kScoreWaves = SGDKV_SCORE_WAVES;  // waves per score workgroup
constexpr int kScoreBlock = 64 * kScoreWaves;

// Opt-in per-kernel timing (see sgdkv_profile_*): brackets a launch with events.
void prof_begin(const char* name, hipStream_t stream);
void prof_end(hipStream_t stream);
#define SGDKV_LAUNCH(name, kernel, grid, block, stream, ...)                  \
  do {                                                                        \
    ::sgdkv::prof_begin(name, stream);                                        \
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);          \
    ::sgdkv::prof_end(stream);                                                \
  } while (0)

// ---------------------------------------------------------------- compress
struct CompressArgs {
  // shapes
  int B, Hq, Hkv, G, D, w, kp, R, dtype;
  int64_t C, s, W, n_scored;  // n_scored = win0: the keys before the window are scored
  int64_t win0;               // position of window row 0; row i sees keys 0..min(win0 + i, C - 1)
  float c2;                   // logit scale * log2(e): scores work in base-2 units
  float out_scale;            // factor on each key's aggregated window sum: 1/G for the means, else 1
  // group aggregation: 0 mean, 1 Ipt. max, 2 Ipt. mean, 3 Ipt. only (see sgdkv.h)
  int agg;
  // per query head q: log2 of its rows' weight (agg 2, 3; -inf for weight 0), or the weight
  // itself (agg 1); unused for agg 0
  float qweight[kMaxIptQHeads];
  // inputs
  const void* q_win;
  const void* k;
  const void* v;
  const float* window_lse;  // natural log, optional
  // outputs
  void* k_out;
  void* v_out;
  int32_t* kept_pos;
  int64_t* offsets;
  float* pooled;  // caller's scores_out or workspace
  // workspace regions
  float* lse_part;  // [B*Hkv][n_lse_chunks][R][2]  (m, s) in base-2 units
  float* lse2;      // [B*Hkv][R]                   base-2 LSE of each window row
  float* colsum;    // [n_rsplit][B*Hkv][n_scored]: one column-sum partial per row split
  uint32_t* hist;   // [B*Hkv][4][256]: histogram of each radix digit
  // [B*Hkv][n_hist_chunks][kChunkHistWords]: per scored chunk, the last digit's histogram of its
  // candidates that match tau's top 24 bits (256 bins), then how many candidates lie above them
  uint32_t* chunk_hist;
  // row splits: the R window rows of a KV head are split over n_rsplit score workgroups per key
  // chunk (grid z), split p holding rows [p*rs_rows, min(R, (p+1)*rs_rows)); rs_rows is a
  // multiple of 16 (of w for the Ipt. max aggregation, so that no query head straddles two)
  int n_rsplit;
  int rs_rows;
  // pass 1's row split: the even one also under Ipt. max (a row's LSE needs no other row, and
  // whole heads would give one split more rows than the others)
  int lse_n_rsplit;
  int lse_rs_rows;
  // chunking
  int64_t score_chunk;  // keys per pass-2 workgroup (multiple of kScoreChunkQuantum)
  // pass 1: n_lse_head chunks of lse_chunk keys over [0, lse_tail0), the keys every window row sees
  // in whole tiles, then (if any key remains that some row sees) one chunk [lse_tail0, min(C, win0 + w))
  // holding the causally masked tiles, which take the exact path
  int64_t lse_chunk;
  int64_t lse_tail0;
  int n_lse_head;
  int n_lse_chunks;     // n_lse_head + the tail chunk
  int n_col_chunks;     // ceil(n_scored / score_chunk)
  int64_t hist_chunk;   // positions per pooling / radix-pass / compaction workgroup (multiple of 256)
  int n_hist_chunks;    // ceil(n_scored / hist_chunk): scored chunks
  int n_cmp_chunks;     // ceil(C / hist_chunk): compaction chunks (the last ones hold window rows only)
  // per KV head of this layer (shared by every sequence)
  int64_t T_layer;
  int64_t m[kMaxKvHeads];           // middle rows kept per head
  int64_t prefix[kMaxKvHeads + 1];  // exclusive prefix sums of the budgets
  int copy_blocks = 0;              // gather work items per segment: ceil(max_h b_h / kCopyRows)
};

hipError_t launch_scores(const CompressArgs& a, hipStream_t stream);      // passes 1 and 2
hipError_t launch_select(const CompressArgs& a, bool scores_only, hipStream_t stream);  // pool .. compact
// The row gather; max_blocks > 0 caps its grid (the copy then runs beside other work).
hipError_t launch_gather(const CompressArgs& a, int max_blocks, hipStream_t stream);

// ------------------------------------------------------------------ decode
struct DecodeArgs {
  int B, Hq, Hkv, G, D, kv_dtype, out_dtype;
  float c2;  // scale * log2(e)
  const void* q;
  const void* k_c;
  const void* v_c;
  const int64_t* offsets;
  int64_t total_rows;  // offsets_host[B*Hkv]: device offsets are clamped to it
  void* out;
  float* lse_out;
  // The splits of a segment are grouped by workgroup (kDecodeWaves splits each), and a workgroup
  // merges its splits into one partial per query head of the group, in its own slot: its flat
  // index in the compact grid, seg * (n_cwg + n_new_wg) + x in the (x, segment) grid. A segment's
  // slots are contiguous (its compressed rows' workgroups, then its appended rows').
  float* part;        // [n_slots][G][D]: o per slot and query head (16-byte aligned rows)
  float* part_ms;     // [n_slots][G][2]: (m, s) per slot and query head
  int64_t chunk;      // rows per split (multiple of 64: at least 128, 256 for batches past two rounds of
                      // 128-row workgroups, or 64 for a batch too small to fill the chip);
                      // on the compact grid it only sizes the workgroups and the appended rows' splits
  int n_chunk_max;    // max over segments of ceil(len / chunk): splits of the compressed rows
  int n_cwg;          // ceil(n_chunk_max / waves per workgroup): workgroups (slots) of the compressed rows; on the
                      // compact grid at least the most any segment was given (appended rows' workgroups follow)
  // rows appended after compression: (b, h) owns rows [0, n_new) of k_new/v_new + (b*Hkv+h)*cap rows;
  // their workgroups come after the compressed ones, at slot n_cwg + j
  const void* k_new;
  const void* v_new;
  int64_t cap, n_new;
  int n_new_chunks;   // ceil(n_new / chunk)
  int64_t n_slots;    // slots the workspace holds (planned for the appended region's capacity)
  // Compact grid (B*Hkv <= kMaxCompactSegs): only workgroups with work are launched, segment
  // after segment (from the host copy of the offsets); segment s owns workgroups
  // [wg_start[s], wg_start[s+1]), its compressed rows' first, then n_new_wg for its appended rows.
  // Otherwise (compact = 0) the grid is (n_cwg + n_new_wg) x segments.
  int compact;
  int n_new_wg;       // ceil(n_new_chunks / waves per workgroup)
  int32_t wg_start[kMaxCompactSegs + 1];
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);

// Static device scratch of the decode entry point that allocates nothing: its size, and the
// current device's address of it (looked up once per device).
constexpr size_t kDecodeScratchBytes = size_t(64) << 20;
hipError_t decode_scratch(void** ptr);
hipError_t launch_append(const DecodeArgs& a, const void* k_step, const void* v_step, void* k_new, void* v_new,
                         int64_t slot, hipStream_t stream);

}  // namespace sgdkv

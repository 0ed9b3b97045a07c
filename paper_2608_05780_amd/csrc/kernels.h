// Kernel launchers (defined in attn.hip and evidence.hip, called from api.hip).
#pragma once
#include <hip/hip_runtime.h>

#include "plan.h"

namespace evisel {

// Device views of the plan tables (one allocation, owned by the mask).
struct DevPlan {
  const BlockDesc* blocks;
  const int32_t* col;
  const BlockDesc* col_desc;  // [nnz] descriptor of each CSR entry's block
  const WorkItem* items;
  const PairedTile* ptile;       // key tiles of paired items
  const BlockDesc* ptile_desc;   // descriptor of each paired tile's block
  const SeqDesc* seqs;
  const TextTile* tiles;
  const int32_t* frame_seq;
  const int32_t* blk_local;  // [nb] local selectable index, -1 for system
  const FramePair* pairs;    // [n_pairs] cross-frame pairs
  const int32_t* ff_out_ptr; // [T+1] pairs whose query frame is t
  const int32_t* ff_out_idx;
  const int32_t* ff_in_ptr;  // [T+1] pairs whose key frame is t
  const int32_t* ff_in_idx;
  int32_t n_pairs;
  int32_t nnz;               // CSR entries
  int32_t n_items, n_tiles, n_seq;
  int32_t S, T, n_text_rows;
  int64_t segtot;
  int32_t hq, hkv, Nv;
  int32_t nb;                // blocks
  int32_t W;                 // history words per row (top-p)
  int32_t hmax;              // longest block history (top-p)
  int32_t topp;              // 1: adaptive top-p retention
};

// Workspace carve-up for one prefill call.
struct Workspace {
  float* pO;     // [slots][64][d]  unnormalised partial outputs
  float* pM;     // [slots][64]     reference max (log2 units)
  float* pL;     // [slots][64]     partial row sums
  float* pNV;    // [slots][64]     log2 partial mass on non-visual keys
  float* seg;    // [hq][segtot]    log2 partial mass per (query row, frame)
  // top-p retention (null for the static rule)
  void* kbar;              // bf16: hi [hkv][d/8][nb][8] then lo; fp32: [hkv][nb][d]
  uint32_t* rbits;         // [hq][nb][W][64] retained history per row
  uint32_t* ubits;         // [hq][nb][W]     union over the block's rows
  float* cpart;            // coarse evidence per-block partial sums
  // frame cues (null unless requested)
  float* segv;             // [hq][nnz][64 / N_v][64] log2 partial mass of a
                           // visual row on each frame of a computed key tile
  float* lse2v;            // [hq][S] log2 LSE of visual rows
  float* intra_part;       // [hkv][T][N_v][N_v] intra-frame sums per kv head
};

struct SelCall {
  const void* q;
  const void* k;
  float scale_log2;        // softmax scale * log2(e)
  float tau;
  int32_t d;
  int32_t fp32;
  uint32_t* rbits;         // outputs (workspace or caller buffers)
  uint32_t* ubits;
};

struct AttnCall {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;            // may be null
  float scale_log2;      // softmax scale * log2(e)
  int32_t d;
  int32_t fp32;          // 1: fp32 inputs/outputs, 0: bf16
  float* segv;           // frame-cue partials of visual rows, or null
  float* lse2v;          // visual rows' log2 LSE, or null
};

hipError_t launch_attention(const DevPlan& p, const Workspace& w,
                            const AttnCall& c, hipStream_t s);
// The software-pipelined attention kernel (attn_pipe.hip): bf16, d = 64 or
// 128, static rule, no frame-cue outputs; launch_attention uses it for
// every call it supports.
bool attention_pipe_supported(const DevPlan& p, const AttnCall& c);
hipError_t launch_attention_pipe(const DevPlan& p, const Workspace& w,
                                 const AttnCall& c, hipStream_t s);
// Top-p retention: mean keys, then per (block, head) the retained history
// of every row (rbits) and the union over the block's rows (ubits).
// LDS bytes the retention kernel needs at its narrowest setting.
size_t select_lds_need(int nh_max, int W);
hipError_t launch_select(const DevPlan& p, const Workspace& w,
                         const SelCall& c, hipStream_t s);
// Coarse query-frame evidence of one layer (top-p masks; the retention
// bits must already be in w.rbits): out [hq][T]. cpart holds
// coarse_part_floats() floats of per-block partial sums.
size_t coarse_part_floats(int n_tiles, int hq, int W);
hipError_t launch_coarse(const DevPlan& p, const Workspace& w,
                         const SelCall& c, float* cpart, float* out,
                         hipStream_t s);
// Sets the per-(row, frame) partial masses to -inf (top-p: key tiles no row
// of a work item retained are skipped and leave no partial).
hipError_t launch_seg_fill(const DevPlan& p, const Workspace& w,
                           hipStream_t s);
// Merge of the split query-token rows (O and LSE into c's outputs), the
// layer's evidence [hq][T] and, when text_mass_layer is not null, the
// query rows' non-visual mass [hq][n_seq], in one launch.
hipError_t launch_combine_evidence(const DevPlan& p, const Workspace& w,
                                   const AttnCall& c, float* evidence_layer,
                                   float* text_mass_layer, hipStream_t s);
hipError_t launch_frame_evidence(const DevPlan& p, const float* evidence,
                                 int32_t n_layers, float* e_qf_layer,
                                 float* e_qf, const int32_t* k_per_seq,
                                 int32_t* topk, hipStream_t s);
// Cross-frame cue of one layer: pairs_out[i] = A_ff of pair i.
hipError_t launch_frame_pairs(const DevPlan& p, const Workspace& w,
                              float* pairs_out, hipStream_t s);
// Intra-frame cue of one layer: out [T][N_v][N_v].
hipError_t launch_intra_frame(const DevPlan& p, const Workspace& w,
                              const AttnCall& c, float* out, hipStream_t s);
// E_ff [n_layers][T] from the cross-frame pairs [n_layers][n_pairs].
hipError_t launch_e_ff(const DevPlan& p, const float* pairs,
                       int32_t n_layers, float* e_ff, hipStream_t s);

}  // namespace evisel

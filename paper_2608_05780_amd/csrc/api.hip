// C ABI of libevisel.so: argument validation, plan upload, launches.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "evisel.h"
#include "kernels.h"
#include "plan.h"

struct evisel_mask {
  evisel::Plan plan;
  void* dev = nullptr;      // one device allocation holding every table
  void* staging = nullptr;  // pinned host copy the upload reads from
  size_t bytes = 0;         // size of both
  size_t items_off = 0;     // offset of the work-item table in both
  hipEvent_t uploaded = nullptr;  // recorded after the last upload copy
  evisel::DevPlan dp{};
  int device = -1;
};

// Workspace of evisel_sparse_prefill_noalloc. Each GPU the library is
// loaded on holds its own copy, at its own address, until the process ends.
// Host code uses this name only to look that address up (scratch_address);
// the name itself is a host-side stand-in, not a device pointer.
static __device__ __align__(256) unsigned char
    scratch[EVISEL_NOALLOC_WORKSPACE_BYTES];

namespace {

thread_local std::string g_err;

evisel_status fail(evisel_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

evisel_status hip_fail(hipError_t e, const char* what) {
  return fail(EVISEL_ERR_HIP,
              std::string(what) + ": " + hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

evisel_status make_plan(const evisel_layout* layout,
                        const evisel_mask_rule* rule, int32_t hq, int32_t hkv,
                        evisel_mask** out, evisel_mask** made) {
  *made = nullptr;
  if (!layout || !rule || !out)
    return fail(EVISEL_ERR_INVALID_ARG, "null layout, rule or out pointer");
  *out = nullptr;
  if (layout->n_seq < 1 || !layout->n_frames || !layout->n_text)
    return fail(EVISEL_ERR_INVALID_ARG,
                "layout needs n_seq >= 1 and n_frames/n_text arrays");
  evisel::Layout L;
  L.Nv = layout->tokens_per_frame;
  L.n_frames.assign(layout->n_frames, layout->n_frames + layout->n_seq);
  L.n_text.assign(layout->n_text, layout->n_text + layout->n_seq);
  if (layout->n_sys)
    L.n_sys.assign(layout->n_sys, layout->n_sys + layout->n_seq);
  evisel::Rule R;
  R.block = rule->block;
  R.sink = rule->sink_blocks;
  R.window = rule->window;
  R.tau = rule->tau_p;
  evisel_mask* m = new (std::nothrow) evisel_mask();
  if (!m) return fail(EVISEL_ERR_NOMEM, "host allocation failed");
  std::string err;
  try {
    err = evisel::build_plan(L, R, hq, hkv, &m->plan);
  } catch (const std::bad_alloc&) {
    delete m;
    return fail(EVISEL_ERR_NOMEM, "host allocation failed");
  }
  if (!err.empty()) {
    delete m;
    return fail(EVISEL_ERR_INVALID_ARG, err);
  }
  if (R.tau > 0.f) {
    const evisel::Plan& P = m->plan;
    const int hmax = P.hist_words * 32;
    if (P.max_item_candidates > evisel::kMaxItemCandidates ||
        evisel::select_lds_need(hmax, P.hist_words) > 160 * 1024) {
      delete m;
      return fail(EVISEL_ERR_UNSUPPORTED,
                  "top-p retention supports at most " +
                      std::to_string(evisel::kMaxItemCandidates) +
                      " candidate key blocks per query block");
    }
  }
  *made = m;
  return EVISEL_OK;
}

template <class T>
size_t put(std::vector<char>& buf, const std::vector<T>& v) {
  const size_t off = align256(buf.size());
  buf.resize(off + align256(v.size() * sizeof(T) + 1));
  if (!v.empty()) std::memcpy(buf.data() + off, v.data(), v.size() * sizeof(T));
  return off;
}

evisel_status upload(evisel_mask* m, hipStream_t s) {
  const evisel::Plan& P = m->plan;
  std::vector<char> buf;
  const size_t o_blk = put(buf, P.blocks), o_col = put(buf, P.col),
               o_cd = put(buf, P.col_desc), o_pt = put(buf, P.ptile),
               o_pd = put(buf, P.ptile_desc), o_it = put(buf, P.items),
               o_seq = put(buf, P.seqs),
               o_tt = put(buf, P.tiles), o_fs = put(buf, P.frame_seq),
               o_bl = put(buf, P.blk_local), o_fp = put(buf, P.pairs),
               o_fop = put(buf, P.ff_out_ptr), o_foi = put(buf, P.ff_out_idx),
               o_fip = put(buf, P.ff_in_ptr), o_fii = put(buf, P.ff_in_idx);
  hipError_t e = hipGetDevice(&m->device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipMalloc(&m->dev, buf.size());
  if (e != hipSuccess) {
    m->dev = nullptr;
    return e == hipErrorOutOfMemory ? fail(EVISEL_ERR_NOMEM, "hipMalloc")
                                    : hip_fail(e, "hipMalloc");
  }
  // The copy reads a pinned staging buffer that the mask keeps until it is
  // freed, so the call returns without waiting for it; the event marks its
  // completion for evisel_mask_free and evisel_mask_permute_work.
  e = hipHostMalloc(&m->staging, buf.size(), hipHostMallocDefault);
  if (e != hipSuccess) {
    m->staging = nullptr;
    return e == hipErrorOutOfMemory ? fail(EVISEL_ERR_NOMEM, "hipHostMalloc")
                                    : hip_fail(e, "hipHostMalloc");
  }
  std::memcpy(m->staging, buf.data(), buf.size());
  m->bytes = buf.size();
  m->items_off = o_it;
  e = hipEventCreateWithFlags(&m->uploaded, hipEventDisableTiming);
  if (e != hipSuccess) {
    m->uploaded = nullptr;
    return hip_fail(e, "hipEventCreate");
  }
  e = hipMemcpyAsync(m->dev, m->staging, buf.size(), hipMemcpyHostToDevice,
                     s);
  if (e == hipSuccess) e = hipEventRecord(m->uploaded, s);
  if (e != hipSuccess) return hip_fail(e, "plan upload");
  char* d = (char*)m->dev;
  evisel::DevPlan& dp = m->dp;
  dp.blocks = (const evisel::BlockDesc*)(d + o_blk);
  dp.col = (const int32_t*)(d + o_col);
  dp.col_desc = (const evisel::BlockDesc*)(d + o_cd);
  dp.ptile = (const evisel::PairedTile*)(d + o_pt);
  dp.ptile_desc = (const evisel::BlockDesc*)(d + o_pd);
  dp.items = (const evisel::WorkItem*)(d + o_it);
  dp.seqs = (const evisel::SeqDesc*)(d + o_seq);
  dp.tiles = (const evisel::TextTile*)(d + o_tt);
  dp.frame_seq = (const int32_t*)(d + o_fs);
  dp.blk_local = (const int32_t*)(d + o_bl);
  dp.pairs = (const evisel::FramePair*)(d + o_fp);
  dp.ff_out_ptr = (const int32_t*)(d + o_fop);
  dp.ff_out_idx = (const int32_t*)(d + o_foi);
  dp.ff_in_ptr = (const int32_t*)(d + o_fip);
  dp.ff_in_idx = (const int32_t*)(d + o_fii);
  dp.n_pairs = (int32_t)P.pairs.size();
  dp.nnz = (int32_t)P.col.size();
  dp.n_items = (int32_t)P.items.size();
  dp.n_tiles = (int32_t)P.tiles.size();
  dp.n_seq = (int32_t)P.seqs.size();
  dp.S = (int32_t)P.S;
  dp.T = (int32_t)P.T;
  dp.n_text_rows = (int32_t)P.n_text_rows;
  dp.segtot = P.segtot;
  dp.hq = P.hq;
  dp.hkv = P.hkv;
  dp.Nv = P.layout.Nv;
  dp.nb = (int32_t)P.blocks.size();
  dp.W = P.hist_words;
  int32_t hmax = 0;
  for (int32_t loc : P.blk_local) hmax = std::max(hmax, loc);
  dp.hmax = hmax;
  dp.topp = P.rule.tau > 0.f ? 1 : 0;
  return EVISEL_OK;
}

struct WsLayout {
  size_t pO, pM, pL, pNV, seg, kbar, rbits, ubits, cpart, total;
  size_t segv, lse2v, intra_part, cue_total;   // frame cues, after `total`
};

WsLayout ws_layout(const evisel::Plan& P, int32_t d) {
  WsLayout w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t rows = (size_t)P.n_slots * 64;
  w.pO = take(rows * d * 4);
  w.pM = take(rows * 4);
  w.pL = take(rows * 4);
  w.pNV = take(rows * 4);
  w.seg = take((size_t)P.hq * P.segtot * 4);
  if (P.rule.tau > 0.f) {
    const size_t nb = P.blocks.size();
    // bf16 keeps hi and lo (2 x 2 bytes), fp32 one float: 4 bytes either way
    w.kbar = take((size_t)P.hkv * nb * d * 4);
    w.rbits = take((size_t)P.hq * nb * P.hist_words * 64 * 4);
    w.ubits = take((size_t)P.hq * nb * P.hist_words * 4);
    w.cpart = take(evisel::coarse_part_floats((int)P.tiles.size(), P.hq,
                                              P.hist_words) * 4);
  } else {
    w.kbar = w.rbits = w.ubits = w.cpart = 0;
  }
  w.total = off;
  const int fpt = P.layout.Nv >= 1 && 64 % P.layout.Nv == 0
                      ? 64 / P.layout.Nv : 1;
  w.segv = take((size_t)P.hq * P.col.size() * fpt * 64 * 4);
  w.lse2v = take((size_t)P.hq * P.S * 4);
  w.intra_part = take((size_t)P.hkv * P.T * P.layout.Nv * P.layout.Nv * 4);
  w.cue_total = off - w.total;
  return w;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

evisel::Workspace carve(const WsLayout& wl, void* workspace, bool topp,
                        bool cues = false) {
  char* wb = (char*)workspace;
  evisel::Workspace w;
  w.pO = (float*)(wb + wl.pO);
  w.pM = (float*)(wb + wl.pM);
  w.pL = (float*)(wb + wl.pL);
  w.pNV = (float*)(wb + wl.pNV);
  w.seg = (float*)(wb + wl.seg);
  w.kbar = topp ? (void*)(wb + wl.kbar) : nullptr;
  w.rbits = topp ? (uint32_t*)(wb + wl.rbits) : nullptr;
  w.ubits = topp ? (uint32_t*)(wb + wl.ubits) : nullptr;
  w.cpart = topp ? (float*)(wb + wl.cpart) : nullptr;
  w.segv = cues ? (float*)(wb + wl.segv) : nullptr;
  w.lse2v = cues ? (float*)(wb + wl.lse2v) : nullptr;
  w.intra_part = cues ? (float*)(wb + wl.intra_part) : nullptr;
  return w;
}

// Checks shared by the compute calls that read q and k.
evisel_status check_qk(const evisel::Plan& P, const void* q, const void* k,
                       int32_t d, evisel_dtype dtype, float softmax_scale,
                       void* workspace, size_t workspace_bytes,
                       const WsLayout& wl) {
  if (!q || !k) return fail(EVISEL_ERR_INVALID_ARG, "null q or k");
  if (!aligned16(q) || !aligned16(k))
    return fail(EVISEL_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  if (!(softmax_scale > 0.f) || softmax_scale > 1e30f)
    return fail(EVISEL_ERR_INVALID_ARG, "softmax_scale must be positive");
  if (d != 64 && d != 128)
    return fail(EVISEL_ERR_UNSUPPORTED, "head dim must be 64 or 128");
  if (dtype != EVISEL_BF16 && dtype != EVISEL_FP32)
    return fail(EVISEL_ERR_UNSUPPORTED, "dtype must be bf16 or fp32");
  if (P.rule.block != 64)
    return fail(EVISEL_ERR_UNSUPPORTED, "attention kernel needs block = 64");
  if (!workspace || workspace_bytes < wl.total)
    return fail(EVISEL_ERR_WORKSPACE,
                "workspace needs " + std::to_string(wl.total) + " bytes");
  if ((uintptr_t)workspace & 255)
    return fail(EVISEL_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return EVISEL_OK;
}

evisel::SelCall sel_call(const void* q, const void* k, int32_t d,
                         evisel_dtype dtype, float softmax_scale, float tau,
                         uint32_t* rbits, uint32_t* ubits) {
  evisel::SelCall c;
  c.q = q;
  c.k = k;
  c.scale_log2 = softmax_scale * 1.4426950408889634f;
  c.tau = tau;
  c.d = d;
  c.fp32 = dtype == EVISEL_FP32;
  c.rbits = rbits;
  c.ubits = ubits;
  return c;
}

// Kernel timing session (evisel_profile_begin / _end).
struct Profile {
  bool open = false;
  bool all = true;             // every kernel, else the attention kernel only
  std::vector<hipEvent_t> ev;  // kProfEvents per timed call
  size_t used = 0;             // calls recorded
  int64_t seen = 0;            // prefill calls since the session began
  int32_t stride = 1;          // calls seen % stride == 0 are recorded
};
Profile g_prof;
constexpr int kProfEvents = 5;
constexpr int kProfAttn = 1;   // events kProfAttn, kProfAttn + 1 bracket K1

void prof_record(size_t call, int k, hipStream_t s) {
  if (!g_prof.all && k != kProfAttn && k != kProfAttn + 1) return;
  (void)hipEventRecord(g_prof.ev[kProfEvents * call + k], s);
}

// Device address of `scratch` per GPU, looked up once per device, with that
// device current, on the first no-allocation call there.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

evisel_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(EVISEL_ERR_UNSUPPORTED,
                "no static workspace for device ordinals above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || ((uintptr_t)p & 255))
      return fail(EVISEL_ERR_HIP, "static workspace is not 256-byte aligned");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return EVISEL_OK;
}

evisel_status check_device(const evisel_mask* m) {
  if (!m) return fail(EVISEL_ERR_INVALID_ARG, "null mask");
  if (!m->dev)
    return fail(EVISEL_ERR_INVALID_ARG,
                "mask has no device copy (built with _host)");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != m->device)
    return fail(EVISEL_ERR_INVALID_ARG,
                "current device differs from the mask's device");
  return EVISEL_OK;
}

}  // namespace

extern "C" {

evisel_status evisel_build_block_mask(const evisel_layout* layout,
                                      const evisel_mask_rule* rule, int32_t hq,
                                      int32_t hkv, void* stream,
                                      evisel_mask** out) {
  evisel_mask* m = nullptr;
  evisel_status st = make_plan(layout, rule, hq, hkv, out, &m);
  if (st != EVISEL_OK) return st;
  st = upload(m, (hipStream_t)stream);
  if (st != EVISEL_OK) {
    evisel_mask_free(m);
    return st;
  }
  *out = m;
  return EVISEL_OK;
}

evisel_status evisel_build_block_mask_host(const evisel_layout* layout,
                                           const evisel_mask_rule* rule,
                                           int32_t hq, int32_t hkv,
                                           evisel_mask** out) {
  evisel_mask* m = nullptr;
  evisel_status st = make_plan(layout, rule, hq, hkv, out, &m);
  if (st != EVISEL_OK) return st;
  *out = m;
  return EVISEL_OK;
}

void evisel_mask_free(evisel_mask* mask) {
  if (!mask) return;
  if (mask->uploaded) {
    (void)hipEventSynchronize(mask->uploaded);   // the copy reads staging
    (void)hipEventDestroy(mask->uploaded);
  }
  if (mask->staging) (void)hipHostFree(mask->staging);
  if (mask->dev) (void)hipFree(mask->dev);
  delete mask;
}

evisel_status evisel_mask_permute_work(evisel_mask* m, const int32_t* perm,
                                       void* stream) {
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  if (!perm) return fail(EVISEL_ERR_INVALID_ARG, "null perm");
  std::vector<evisel::WorkItem>& it = m->plan.items;
  const size_t n = it.size();
  std::vector<char> seen(n, 0);
  for (size_t i = 0; i < n; ++i) {
    if (perm[i] < 0 || (size_t)perm[i] >= n || seen[perm[i]])
      return fail(EVISEL_ERR_INVALID_ARG,
                  "perm is not a permutation of the work items");
    seen[perm[i]] = 1;
  }
  std::vector<evisel::WorkItem> next(n);
  for (size_t i = 0; i < n; ++i) next[i] = it[perm[i]];
  // the previous upload may still read the staging buffer
  hipError_t e = hipEventSynchronize(m->uploaded);
  if (e != hipSuccess) return hip_fail(e, "plan upload wait");
  it.swap(next);
  char* st_items = (char*)m->staging + m->items_off;
  if (n) std::memcpy(st_items, it.data(), n * sizeof(evisel::WorkItem));
  hipStream_t s = (hipStream_t)stream;
  e = hipMemcpyAsync((char*)m->dev + m->items_off, st_items,
                     n * sizeof(evisel::WorkItem), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipEventRecord(m->uploaded, s);
  if (e != hipSuccess) return hip_fail(e, "work list upload");
  return EVISEL_OK;
}

evisel_status evisel_mask_info(const evisel_mask* m, evisel_mask_stats* out) {
  if (!m || !out) return fail(EVISEL_ERR_INVALID_ARG, "null argument");
  const evisel::Plan& P = m->plan;
  out->n_tokens = P.S;
  out->n_frames_total = P.T;
  out->n_text_rows = P.n_text_rows;
  out->n_blocks = (int64_t)P.blocks.size();
  out->n_active_pairs = (int64_t)P.col.size();
  out->n_work_items = (int64_t)P.items.size();
  out->n_text_tiles = (int64_t)P.tiles.size();
  out->n_chunk_slots = P.n_slots;
  out->hq = P.hq;
  out->hkv = P.hkv;
  out->block = P.rule.block;
  out->tokens_per_frame = P.layout.Nv;
  out->hist_words = P.hist_words;
  out->tau_p = P.rule.tau;
  out->n_frame_pairs = (int64_t)P.pairs.size();
  out->n_paired_tiles = (int64_t)P.ptile.size();
  return EVISEL_OK;
}

evisel_status evisel_mask_export(const evisel_mask* m, int32_t* blk_start,
                                 int32_t* blk_len, int32_t* blk_region,
                                 int32_t* blk_video, int32_t* row_ptr,
                                 int32_t* col) {
  if (!m) return fail(EVISEL_ERR_INVALID_ARG, "null mask");
  const evisel::Plan& P = m->plan;
  for (size_t b = 0; b < P.blocks.size(); ++b) {
    if (blk_start) blk_start[b] = P.blocks[b].start;
    if (blk_len) blk_len[b] = P.blocks[b].len;
    if (blk_region) blk_region[b] = P.blocks[b].region;
  }
  if (blk_video) {
    size_t b = 0;
    for (size_t n = 0; n < P.seqs.size(); ++n)
      while (b < P.blocks.size() && P.blocks[b].start < P.seqs[n].end)
        blk_video[b++] = (int32_t)n;
  }
  if (row_ptr)
    std::memcpy(row_ptr, P.row_ptr.data(), P.row_ptr.size() * 4);
  if (col && !P.col.empty()) std::memcpy(col, P.col.data(), P.col.size() * 4);
  return EVISEL_OK;
}

evisel_status evisel_mask_export_work(const evisel_mask* m, int32_t* qblock,
                                      int32_t* head, int32_t* nheads,
                                      int32_t* kb_begin, int32_t* kb_end,
                                      int32_t* slot, int32_t* qblock2,
                                      int32_t* slot2) {
  if (!m) return fail(EVISEL_ERR_INVALID_ARG, "null mask");
  const auto& it = m->plan.items;
  for (size_t i = 0; i < it.size(); ++i) {
    if (qblock) qblock[i] = it[i].qblock;
    if (head) head[i] = it[i].head;
    if (nheads) nheads[i] = it[i].nheads;
    if (kb_begin) kb_begin[i] = it[i].kb_begin;
    if (kb_end) kb_end[i] = it[i].kb_end;
    if (slot) slot[i] = it[i].slot;
    if (qblock2) qblock2[i] = it[i].qblock2;
    if (slot2) slot2[i] = it[i].slot2;
  }
  return EVISEL_OK;
}

evisel_status evisel_mask_export_paired(const evisel_mask* m, int32_t* block,
                                        int32_t* pos_a, int32_t* pos_b) {
  if (!m) return fail(EVISEL_ERR_INVALID_ARG, "null mask");
  const auto& pt = m->plan.ptile;
  for (size_t i = 0; i < pt.size(); ++i) {
    if (block) block[i] = pt[i].block;
    if (pos_a) pos_a[i] = pt[i].pos[0];
    if (pos_b) pos_b[i] = pt[i].pos[1];
  }
  return EVISEL_OK;
}

size_t evisel_sparse_prefill_workspace(const evisel_mask* m, int32_t d) {
  if (!m || (d != 64 && d != 128)) return 0;
  return ws_layout(m->plan, d).total;
}

evisel_status evisel_sparse_prefill(const evisel_mask* m, int32_t layer,
                                    int32_t n_layers, const void* q,
                                    const void* k, const void* v, int32_t d,
                                    evisel_dtype dtype, float softmax_scale,
                                    void* out, float* lse, float* evidence,
                                    float* text_mass, float* frame_pairs,
                                    float* intra_frame, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  const evisel::Plan& P = m->plan;
  if (n_layers < 1 || layer < 0 || layer >= n_layers)
    return fail(EVISEL_ERR_INVALID_ARG, "need 0 <= layer < n_layers");
  if (!v || !out || !evidence)
    return fail(EVISEL_ERR_INVALID_ARG, "null v, out or evidence");
  if (!aligned16(v) || !aligned16(out))
    return fail(EVISEL_ERR_INVALID_ARG, "v and out must be 16-byte aligned");
  const WsLayout wl = ws_layout(P, d);
  st = check_qk(P, q, k, d, dtype, softmax_scale, workspace, workspace_bytes,
                wl);
  if (st != EVISEL_OK) return st;
  const int nv = P.layout.Nv;
  if (nv < 8 || 64 % nv != 0)
    return fail(EVISEL_ERR_UNSUPPORTED,
                "tokens_per_frame must divide 64 and be >= 8");
  const bool topp = P.rule.tau > 0.f;
  const bool cues = frame_pairs || intra_frame;
  if (cues && workspace_bytes < wl.total + wl.cue_total)
    return fail(EVISEL_ERR_WORKSPACE,
                "frame cues need " + std::to_string(wl.total + wl.cue_total) +
                    " bytes of workspace");
  if (cues && ((uintptr_t)frame_pairs & 3 || (uintptr_t)intra_frame & 3))
    return fail(EVISEL_ERR_INVALID_ARG, "cue outputs must be 4-byte aligned");
  const evisel::Workspace w = carve(wl, workspace, topp, cues);
  evisel::AttnCall c;
  c.q = q;
  c.k = k;
  c.v = v;
  c.o = out;
  c.lse = lse;
  c.scale_log2 = softmax_scale * 1.4426950408889634f;
  c.d = d;
  c.fp32 = dtype == EVISEL_FP32;
  c.segv = frame_pairs ? w.segv : nullptr;
  c.lse2v = cues ? w.lse2v : nullptr;
  hipStream_t s = (hipStream_t)stream;
  const bool prof = g_prof.open && g_prof.seen++ % g_prof.stride == 0 &&
                    g_prof.used < g_prof.ev.size() / kProfEvents;
  const size_t call = g_prof.used;
  if (prof) prof_record(call, 0, s);
  hipError_t e = hipSuccess;
  if (topp) {
    e = evisel::launch_select(
        m->dp, w,
        sel_call(q, k, d, dtype, softmax_scale, P.rule.tau, w.rbits, w.ubits),
        s);
    if (e != hipSuccess) return hip_fail(e, "retention launch");
    e = evisel::launch_seg_fill(m->dp, w, s);
    if (e != hipSuccess) return hip_fail(e, "partial-mass fill launch");
  }
  if (prof) prof_record(call, 1, s);
  e = evisel::launch_attention(m->dp, w, c, s);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  if (prof) prof_record(call, 2, s);
  e = evisel::launch_combine_evidence(
      m->dp, w, c, evidence + (size_t)layer * P.hq * P.T,
      text_mass ? text_mass + (size_t)layer * P.hq * P.seqs.size() : nullptr,
      s);
  if (e != hipSuccess) return hip_fail(e, "combine and evidence launch");
  if (prof) prof_record(call, 3, s);
  if (frame_pairs) {
    e = evisel::launch_frame_pairs(
        m->dp, w, frame_pairs + (size_t)layer * P.pairs.size(), s);
    if (e != hipSuccess) return hip_fail(e, "frame pair launch");
  }
  if (intra_frame) {
    const size_t nv = (size_t)P.layout.Nv;
    e = evisel::launch_intra_frame(
        m->dp, w, c, intra_frame + (size_t)layer * P.T * nv * nv, s);
    if (e != hipSuccess) return hip_fail(e, "intra-frame launch");
  }
  if (prof) {
    prof_record(call, 4, s);
    g_prof.used++;
  }
  return EVISEL_OK;
}

evisel_status evisel_sparse_prefill_noalloc(
    const evisel_mask* m, int32_t layer, int32_t n_layers, const void* q,
    const void* k, const void* v, int32_t d, evisel_dtype dtype,
    float softmax_scale, void* out, float* lse, float* evidence,
    float* text_mass, float* frame_pairs, float* intra_frame, void* stream) {
  // the mask's device is the current one (checked), so the lookup below
  // runs with the right device current
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  if (d == 64 || d == 128) {
    const WsLayout wl = ws_layout(m->plan, d);
    const size_t need =
        wl.total + (frame_pairs || intra_frame ? wl.cue_total : 0);
    if (need > EVISEL_NOALLOC_WORKSPACE_BYTES)
      return fail(EVISEL_ERR_WORKSPACE,
                  "this mask needs " + std::to_string(need) +
                      " bytes of workspace; the static workspace holds " +
                      std::to_string(EVISEL_NOALLOC_WORKSPACE_BYTES));
  }
  void* ws = nullptr;
  st = scratch_address(m->device, &ws);
  if (st != EVISEL_OK) return st;
  // the ordinary entry point with that workspace: it allocates nothing and
  // no kernel reads workspace bytes the same call has not written
  return evisel_sparse_prefill(m, layer, n_layers, q, k, v, d, dtype,
                               softmax_scale, out, lse, evidence, text_mass,
                               frame_pairs, intra_frame, ws,
                               EVISEL_NOALLOC_WORKSPACE_BYTES, stream);
}

size_t evisel_cue_workspace(const evisel_mask* m, int32_t d) {
  if (!m || (d != 64 && d != 128)) return 0;
  return ws_layout(m->plan, d).cue_total;
}

evisel_status evisel_mask_export_pairs(const evisel_mask* m, int32_t* a,
                                       int32_t* b) {
  if (!m) return fail(EVISEL_ERR_INVALID_ARG, "null mask");
  const auto& pr = m->plan.pairs;
  for (size_t i = 0; i < pr.size(); ++i) {
    if (a) a[i] = pr[i].a;
    if (b) b[i] = pr[i].b;
  }
  return EVISEL_OK;
}

evisel_status evisel_coarse_evidence(const evisel_mask* m, const void* q,
                                     const void* k, int32_t d,
                                     evisel_dtype dtype, float softmax_scale,
                                     float* evidence, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  const evisel::Plan& P = m->plan;
  if (!(P.rule.tau > 0.f))
    return fail(EVISEL_ERR_INVALID_ARG,
                "the coarse map needs a top-p mask (tau_p > 0)");
  if (!evidence || ((uintptr_t)evidence & 3))
    return fail(EVISEL_ERR_INVALID_ARG, "null or misaligned evidence");
  const WsLayout wl = ws_layout(P, d);
  st = check_qk(P, q, k, d, dtype, softmax_scale, workspace, workspace_bytes,
                wl);
  if (st != EVISEL_OK) return st;
  const evisel::Workspace w = carve(wl, workspace, true);
  const evisel::SelCall c = sel_call(q, k, d, dtype, softmax_scale,
                                     P.rule.tau, w.rbits, w.ubits);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = evisel::launch_select(m->dp, w, c, s);
  if (e != hipSuccess) return hip_fail(e, "retention launch");
  e = evisel::launch_coarse(m->dp, w, c, w.cpart, evidence, s);
  if (e != hipSuccess) return hip_fail(e, "coarse evidence launch");
  return EVISEL_OK;
}

evisel_status evisel_select_blocks(const evisel_mask* m, const void* q,
                                   const void* k, int32_t d,
                                   evisel_dtype dtype, float softmax_scale,
                                   uint32_t* row_bits, uint32_t* block_bits,
                                   void* workspace, size_t workspace_bytes,
                                   void* stream) {
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  const evisel::Plan& P = m->plan;
  if (!(P.rule.tau > 0.f))
    return fail(EVISEL_ERR_INVALID_ARG,
                "mask was built without top-p retention (tau_p = 0)");
  if (!row_bits || !block_bits)
    return fail(EVISEL_ERR_INVALID_ARG, "null row_bits or block_bits");
  if (((uintptr_t)row_bits & 3) || ((uintptr_t)block_bits & 3))
    return fail(EVISEL_ERR_INVALID_ARG, "bit arrays must be 4-byte aligned");
  const WsLayout wl = ws_layout(P, d);
  st = check_qk(P, q, k, d, dtype, softmax_scale, workspace, workspace_bytes,
                wl);
  if (st != EVISEL_OK) return st;
  const evisel::Workspace w = carve(wl, workspace, true);
  hipError_t e = evisel::launch_select(
      m->dp, w,
      sel_call(q, k, d, dtype, softmax_scale, P.rule.tau, row_bits,
               block_bits),
      (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "retention launch");
  return EVISEL_OK;
}

evisel_status evisel_frame_evidence(const evisel_mask* m,
                                    const float* evidence, int32_t n_layers,
                                    float* e_qf_layer, float* e_qf,
                                    const int32_t* k_per_seq,
                                    int32_t* topk_idx,
                                    const float* frame_pairs, float* e_ff,
                                    void* stream) {
  evisel_status st = check_device(m);
  if (st != EVISEL_OK) return st;
  if (!evidence || !e_qf || n_layers < 1)
    return fail(EVISEL_ERR_INVALID_ARG, "null evidence/e_qf or n_layers < 1");
  if (k_per_seq && !topk_idx)
    return fail(EVISEL_ERR_INVALID_ARG, "k_per_seq given without topk_idx");
  if (k_per_seq)
    for (const auto& sq : m->plan.seqs)
      if (sq.n_frames > 65536)
        return fail(EVISEL_ERR_UNSUPPORTED,
                    "top-k supports at most 65536 frames per video");
  if (e_ff && !frame_pairs)
    return fail(EVISEL_ERR_INVALID_ARG, "e_ff needs frame_pairs");
  hipError_t e = evisel::launch_frame_evidence(m->dp, evidence, n_layers,
                                               e_qf_layer, e_qf, k_per_seq,
                                               topk_idx, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "frame evidence launch");
  if (e_ff) {
    e = evisel::launch_e_ff(m->dp, frame_pairs, n_layers, e_ff,
                            (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "e_ff launch");
  }
  return EVISEL_OK;
}

evisel_status evisel_profile_begin(int32_t capacity, int32_t all_kernels,
                                   int32_t stride) {
  if (capacity < 1) return fail(EVISEL_ERR_INVALID_ARG, "capacity < 1");
  if (stride < 1) return fail(EVISEL_ERR_INVALID_ARG, "stride < 1");
  if (g_prof.open)
    return fail(EVISEL_ERR_INVALID_ARG, "a profiling session is open");
  g_prof = Profile();
  g_prof.all = all_kernels != 0;
  g_prof.stride = stride;
  try {
    g_prof.ev.resize((size_t)capacity * kProfEvents);
  } catch (const std::bad_alloc&) {
    return fail(EVISEL_ERR_NOMEM, "host allocation failed");
  }
  for (size_t i = 0; i < g_prof.ev.size(); ++i) {
    hipError_t e = hipEventCreate(&g_prof.ev[i]);
    if (e != hipSuccess) {
      for (size_t j = 0; j < i; ++j) (void)hipEventDestroy(g_prof.ev[j]);
      g_prof = Profile();
      return hip_fail(e, "hipEventCreate");
    }
  }
  g_prof.open = true;
  return EVISEL_OK;
}

evisel_status evisel_profile_end(double* ms, int64_t* n_calls) {
  if (!g_prof.open)
    return fail(EVISEL_ERR_INVALID_ARG, "no profiling session is open");
  constexpr int kSpans = kProfEvents - 1;
  double acc[kSpans] = {};
  hipError_t err = hipSuccess;
  for (size_t c = 0; c < g_prof.used && err == hipSuccess; ++c) {
    const hipEvent_t* ev = &g_prof.ev[kProfEvents * c];
    const int k0 = g_prof.all ? 0 : kProfAttn;
    const int k1 = g_prof.all ? kSpans : kProfAttn + 1;
    err = hipEventSynchronize(ev[k1]);
    for (int k = k0; k < k1 && err == hipSuccess; ++k) {
      float t = 0.f;
      err = hipEventElapsedTime(&t, ev[k], ev[k + 1]);
      acc[k] += t;
    }
  }
  const int64_t used = (int64_t)g_prof.used;
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof = Profile();
  if (err != hipSuccess) return hip_fail(err, "profile events");
  if (ms)
    for (int k = 0; k < kSpans; ++k) ms[k] = acc[k];
  if (n_calls) *n_calls = used;
  return EVISEL_OK;
}

const char* evisel_last_error(void) { return g_err.c_str(); }

}  // extern "C"

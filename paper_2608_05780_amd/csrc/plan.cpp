// Host plan builder: block partition, active block pairs, work list.
//
// Blocks follow the frame-aligned partition of the paper's appendix
// ("Detailed Sparse Prefilling"): every region of every video (system prefix,
// visual tokens, query tokens) is cut into blocks of B tokens from the
// region's start, the last one possibly short, and no block crosses a video.
// Active pairs follow the static rule of evisel_mask_rule: the system prefix
// is always visible, a visual block keeps the sink blocks, `window` preceding
// blocks and itself, a query-token block keeps every visual block and the
// query-token blocks up to itself.
#include "plan.h"

#include <algorithm>
#include <limits>
#include <map>
#include <numeric>

namespace evisel {
namespace {

struct Item {
  WorkItem w;
  int64_t cost;
  int64_t group = 0;   // query-token items: (video, kv head, chunk)
};

}  // namespace

std::string build_plan(const Layout& L, const Rule& R, int32_t hq, int32_t hkv,
                       Plan* out) {
  const size_t nseq = L.n_frames.size();
  if (nseq == 0) return "layout has no video";
  if (L.n_text.size() != nseq || (!L.n_sys.empty() && L.n_sys.size() != nseq))
    return "layout arrays differ in length";
  if (L.Nv < 1) return "tokens_per_frame must be >= 1";
  if (R.block < 1) return "block must be >= 1";
  if (R.sink < 0) return "sink_blocks must be >= 0";
  if (R.window < -1) return "window must be >= 0 or -1";
  if (!(R.tau >= 0.f && R.tau <= 1.f)) return "tau_p must be in [0, 1]";
  if (hq < 1 || hkv < 1 || hq % hkv != 0)
    return "head counts must satisfy hq >= 1, hkv >= 1, hq % hkv == 0";
  if (hq > 4096) return "hq too large";

  Plan& P = *out;
  P = Plan();
  P.layout = L;
  if (P.layout.n_sys.empty()) P.layout.n_sys.assign(nseq, 0);
  P.rule = R;
  const bool topp = R.tau > 0.f;
  // top-p: every causal block is a candidate
  const int32_t window = topp ? -1 : R.window;
  P.hq = hq;
  P.hkv = hkv;

  // ---- videos and blocks -------------------------------------------------
  int64_t tok = 0, frame = 0, trow = 0, segbase = 0;
  std::vector<std::vector<int32_t>> sysb(nseq), visb(nseq), txtb(nseq);
  for (size_t n = 0; n < nseq; ++n) {
    const int64_t ns = P.layout.n_sys[n], nf = L.n_frames[n], nt = L.n_text[n];
    if (ns < 0 || nf < 1 || nt < 1)
      return "video " + std::to_string(n) +
             ": need n_sys >= 0, n_frames >= 1, n_text >= 1";
    const int64_t nvis = nf * L.Nv;
    SeqDesc s{};
    s.tok0 = (int32_t)tok;
    s.vis0 = (int32_t)(tok + ns);
    s.txt0 = (int32_t)(tok + ns + nvis);
    const int64_t end = tok + ns + nvis + nt;
    if (end >= (int64_t(1) << 31) - 64) return "too many tokens (>= 2^31)";
    s.end = (int32_t)end;
    s.frame0 = (int32_t)frame;
    s.n_frames = (int32_t)nf;
    s.textrow0 = (int32_t)trow;
    s.n_text = (int32_t)nt;
    s.segbase = segbase;
    auto cut = [&](int64_t a, int64_t e, int32_t reg,
                   std::vector<int32_t>& ids) {
      for (int64_t b = a; b < e; b += R.block) {
        BlockDesc d{};
        d.start = (int32_t)b;
        d.len = (int32_t)std::min<int64_t>(R.block, e - b);
        d.region = reg;
        d.aux = reg == kVis   ? (int32_t)(frame + (b - s.vis0) / L.Nv)
                : reg == kTxt ? (int32_t)(trow + (b - s.txt0))
                              : -1;
        ids.push_back((int32_t)P.blocks.size());
        P.blocks.push_back(d);
      }
    };
    cut(s.tok0, s.vis0, kSys, sysb[n]);
    cut(s.vis0, s.txt0, kVis, visb[n]);
    cut(s.txt0, s.end, kTxt, txtb[n]);
    P.seqs.push_back(s);
    for (int64_t f = 0; f < nf; ++f) P.frame_seq.push_back((int32_t)n);
    tok = end;
    frame += nf;
    trow += nt;
    segbase += nt * nf;
  }
  P.S = tok;
  P.T = frame;
  P.n_text_rows = trow;
  P.segtot = segbase;

  // ---- CSR of active pairs ----------------------------------------------
  const int32_t nb = (int32_t)P.blocks.size();
  P.row_ptr.assign(nb + 1, 0);
  std::vector<int32_t> rowlist;
  for (size_t n = 0; n < nseq; ++n) {
    const auto &sb = sysb[n], &vb = visb[n], &tb = txtb[n];
    for (size_t j = 0; j < sb.size(); ++j) {   // system rows: causal prefix
      rowlist.assign(sb.begin(), sb.begin() + j + 1);
      P.row_ptr[sb[j] + 1] = (int32_t)rowlist.size();
      P.col.insert(P.col.end(), rowlist.begin(), rowlist.end());
    }
    const int32_t nvb = (int32_t)vb.size();
    for (int32_t i = 0; i < nvb; ++i) {        // visual rows
      rowlist.assign(sb.begin(), sb.end());
      const int32_t lo = window < 0 ? 0 : std::max(0, i - window);
      for (int32_t b = 0; b < std::min(R.sink, lo); ++b)
        rowlist.push_back(vb[b]);
      for (int32_t b = lo; b <= i; ++b) rowlist.push_back(vb[b]);
      P.row_ptr[vb[i] + 1] = (int32_t)rowlist.size();
      P.col.insert(P.col.end(), rowlist.begin(), rowlist.end());
    }
    for (size_t t = 0; t < tb.size(); ++t) {   // query-token rows: dense
      rowlist.assign(sb.begin(), sb.end());
      rowlist.insert(rowlist.end(), vb.begin(), vb.end());
      rowlist.insert(rowlist.end(), tb.begin(), tb.begin() + t + 1);
      P.row_ptr[tb[t] + 1] = (int32_t)rowlist.size();
      P.col.insert(P.col.end(), rowlist.begin(), rowlist.end());
    }
  }
  // row_ptr currently holds row lengths at [b+1]; blocks are numbered in
  // token order and rows were appended in the same order, so a prefix sum
  // gives the offsets.
  for (int32_t b = 0; b < nb; ++b) P.row_ptr[b + 1] += P.row_ptr[b];
  if ((int64_t)P.row_ptr[nb] != (int64_t)P.col.size())
    return "internal error: CSR size mismatch";
  P.col_desc.resize(P.col.size());
  for (size_t p = 0; p < P.col.size(); ++p) P.col_desc[p] = P.blocks[P.col[p]];

  // ---- selectable blocks (top-p bookkeeping) -------------------------------
  P.blk_local.assign(nb, -1);
  int32_t max_sel = 0;
  for (size_t n = 0; n < nseq; ++n) {
    int32_t j = 0;
    for (int32_t b : visb[n]) P.blk_local[b] = j++;
    for (int32_t b : txtb[n]) P.blk_local[b] = j++;
    max_sel = std::max(max_sel, j);
  }
  // bits for history blocks 0 .. max_sel - 2
  P.hist_words = std::max(1, (max_sel - 1 + 31) / 32);

  // ---- frame pairs of the cross-frame cue ---------------------------------
  for (size_t n = 0; n < nseq; ++n) {
    const int64_t vis0 = P.seqs[n].vis0, frame0 = P.seqs[n].frame0;
    for (int32_t qb : visb[n]) {
      const BlockDesc& q = P.blocks[qb];
      const int32_t fa0 = (int32_t)((q.start - vis0) / L.Nv);
      const int32_t fa1 = (int32_t)((q.start + q.len - 1 - vis0) / L.Nv);
      for (int32_t p = P.row_ptr[qb]; p < P.row_ptr[qb + 1]; ++p) {
        const BlockDesc& k = P.blocks[P.col[p]];
        if (k.region != kVis) continue;
        const int32_t fb0 = (int32_t)((k.start - vis0) / L.Nv);
        const int32_t fb1 = (int32_t)((k.start + k.len - 1 - vis0) / L.Nv);
        for (int32_t fa = fa0; fa <= fa1; ++fa)
          for (int32_t fb = fb0; fb <= fb1 && fb < fa; ++fb) {
            FramePair fp;
            fp.pos = p;
            fp.a = (int32_t)(frame0 + fa);
            fp.b = (int32_t)(frame0 + fb);
            fp.qblock = qb;
            fp.roff = (int32_t)(vis0 + (int64_t)fa * L.Nv - q.start);
            fp.koff = fb - fb0;
            P.pairs.push_back(fp);
          }
      }
    }
  }
  auto index_by = [&](bool by_a, std::vector<int32_t>& ptr,
                      std::vector<int32_t>& idx) {
    ptr.assign(P.T + 1, 0);
    for (const FramePair& fp : P.pairs) ptr[(by_a ? fp.a : fp.b) + 1]++;
    for (int64_t t = 0; t < P.T; ++t) ptr[t + 1] += ptr[t];
    idx.assign(P.pairs.size(), 0);
    std::vector<int32_t> fill(ptr.begin(), ptr.end() - 1);
    for (size_t i = 0; i < P.pairs.size(); ++i)
      idx[fill[by_a ? P.pairs[i].a : P.pairs[i].b]++] = (int32_t)i;
  };
  index_by(true, P.ff_out_ptr, P.ff_out_idx);
  index_by(false, P.ff_in_ptr, P.ff_in_idx);

  // ---- work items ---------------------------------------------------------
  const int32_t group = hq / hkv;
  const int32_t pairs = (group + kHeadsPerItem - 1) / kHeadsPerItem;
  int64_t total = 0;
  for (int32_t b = 0; b < nb; ++b)
    total += (int64_t)(P.row_ptr[b + 1] - P.row_ptr[b] + 1) * hkv * pairs;
  const int64_t avg = (total + kTargetSlots - 1) / kTargetSlots;
  P.chunk_blocks = (int32_t)std::max<int64_t>(16, avg);

  // Paired items: the kv group's odd head takes two query blocks in one
  // item. Both CSR rows are in ascending key-block order, so their runs
  // merge by key block. (Under top-p each half skips the history blocks its
  // own rows did not retain.)
  auto paired = [&](int32_t qa, int32_t a0, int32_t a1, int32_t qb2,
                    int32_t c0, int32_t c1, int32_t h, int32_t slot_a,
                    int32_t slot_b, int32_t n, int32_t nch) {
    const int32_t begin = (int32_t)P.ptile.size();
    const int32_t none = std::numeric_limits<int32_t>::max();
    int32_t i = a0, j = c0;
    while (i < a1 || j < c1) {
      const int32_t ka = i < a1 ? P.col[i] : none;
      const int32_t kb = j < c1 ? P.col[j] : none;
      PairedTile t;
      t.block = std::min(ka, kb);
      t.pos[0] = ka == t.block ? i++ : -1;
      t.pos[1] = kb == t.block ? j++ : -1;
      P.ptile.push_back(t);
    }
    return WorkItem{qa, h,     1,  begin, (int32_t)P.ptile.size(),
                    slot_a, n, nch, qb2,  slot_b};
  };

  std::vector<Item> txt_items, other_items;
  for (size_t n = 0; n < nseq; ++n) {
    // query-token tiles of this video and their chunk slots
    struct Tile {
      int32_t b, rb, len, nch, slot0;
    };
    std::vector<Tile> vt;
    for (int32_t b : txtb[n]) {
      const int32_t rb = P.row_ptr[b], len = P.row_ptr[b + 1] - rb;
      const int32_t nch = (len + P.chunk_blocks - 1) / P.chunk_blocks;
      TextTile tt{b, (int32_t)n, nch, (int32_t)P.n_slots};
      if (P.seqs[n].n_tiles == 0) P.seqs[n].tile0 = (int32_t)P.tiles.size();
      P.seqs[n].n_tiles++;
      P.tiles.push_back(tt);
      vt.push_back({b, rb, len, nch, tt.slot0});
      P.n_slots += (int64_t)hq * nch;
    }
    // equal-size chunks: chunk c of a tile covers [rb + c*len/nch, ...)
    auto lo = [](const Tile& t, int32_t c) {
      return t.rb + (int32_t)((int64_t)c * t.len / t.nch);
    };
    for (size_t ti = 0; ti < vt.size(); ++ti) {
      const Tile& t = vt[ti];
      for (int32_t g = 0; g < hkv; ++g)
        for (int32_t pp = 0; pp < pairs; ++pp) {
          const int32_t h0 = g * group + pp * kHeadsPerItem;
          const int32_t nh = std::min(kHeadsPerItem, group - pp * kHeadsPerItem);
          const bool pr = nh == 1;
          // odd head: chunk c of tiles 2i and 2i+1 share one item
          const int32_t c_first =
              pr && ti % 2 == 1 ? std::min(vt[ti - 1].nch, t.nch) : 0;
          for (int32_t c = c_first; c < t.nch; ++c) {
            const int64_t key = ((int64_t)n * hkv + g) * 65536 + c;
            if (pr && ti % 2 == 0 && ti + 1 < vt.size() &&
                c < vt[ti + 1].nch) {
              const Tile& u = vt[ti + 1];
              const WorkItem w = paired(
                  t.b, lo(t, c), lo(t, c + 1), u.b, lo(u, c), lo(u, c + 1),
                  h0, t.slot0 + h0 * t.nch + c, u.slot0 + h0 * u.nch + c,
                  (int32_t)n, t.nch);
              txt_items.push_back({w, w.kb_end - w.kb_begin + 1, key});
              continue;
            }
            const WorkItem w{t.b, h0, nh, lo(t, c), lo(t, c + 1),
                             t.slot0 + h0 * t.nch + c, (int32_t)n, t.nch,
                             -1, -1};
            txt_items.push_back({w, w.kb_end - w.kb_begin + 1, key});
          }
        }
    }
    // visual and system rows, ordered by (kv head, block, head pair) so that
    // neighbouring launches share key/value tiles
    for (int32_t g = 0; g < hkv; ++g) {
      auto add = [&](const std::vector<int32_t>& ids) {
        for (size_t i = 0; i < ids.size(); ++i) {
          const int32_t b = ids[i];
          for (int32_t pp = 0; pp < pairs; ++pp) {
            const int32_t h0 = g * group + pp * kHeadsPerItem;
            const int32_t nh =
                std::min(kHeadsPerItem, group - pp * kHeadsPerItem);
            if (nh == 1) {
              // odd head: blocks 2i and 2i+1 of the region share one item
              if (i % 2 == 1) continue;
              if (i + 1 < ids.size()) {
                const int32_t b2 = ids[i + 1];
                const WorkItem w =
                    paired(b, P.row_ptr[b], P.row_ptr[b + 1], b2,
                           P.row_ptr[b2], P.row_ptr[b2 + 1], h0, -1, -1,
                           (int32_t)n, 0);
                other_items.push_back({w, w.kb_end - w.kb_begin + 1});
                continue;
              }
            }
            const WorkItem w{b, h0, nh, P.row_ptr[b], P.row_ptr[b + 1], -1,
                             (int32_t)n, 0, -1, -1};
            other_items.push_back({w, P.row_ptr[b + 1] - P.row_ptr[b] + 1});
          }
        }
      };
      add(sysb[n]);
      add(visb[n]);
    }
  }
  P.ptile_desc.resize(P.ptile.size());
  for (size_t i = 0; i < P.ptile.size(); ++i)
    P.ptile_desc[i] = P.blocks[P.ptile[i].block];

  // Longest-first over the XCD queues: split query-token items go first, by
  // LPT; the remaining items keep their locality order and are cut into
  // contiguous runs that level the queues.
  // Query-token items that read the same key range (same video, kv head
  // and chunk) go to one XCD together, so that its L2 fetches the range
  // once; the groups are balanced longest-first over the XCDs.
  std::map<int64_t, std::vector<Item>> groups;
  for (const Item& it : txt_items) groups[it.group].push_back(it);
  std::vector<std::pair<int64_t, int64_t>> gcost;   // (cost, key)
  for (auto& kv : groups) {
    int64_t c = 0;
    for (const Item& it : kv.second) c += it.cost;
    gcost.push_back({c, kv.first});
  }
  std::stable_sort(gcost.begin(), gcost.end(),
                   [](const std::pair<int64_t, int64_t>& a,
                      const std::pair<int64_t, int64_t>& b) {
                     return a.first > b.first;
                   });
  std::vector<std::vector<WorkItem>> q(kXcds);
  std::vector<int64_t> load(kXcds, 0);
  for (const auto& gc : gcost) {
    const int x = (int)(std::min_element(load.begin(), load.end()) -
                        load.begin());
    for (const Item& it : groups[gc.second]) q[x].push_back(it.w);
    load[x] += gc.first;
  }
  int64_t rest = 0;
  for (const Item& it : other_items) rest += it.cost;
  const int64_t all = rest + std::accumulate(load.begin(), load.end(),
                                             int64_t(0));
  const int64_t target = (all + kXcds - 1) / kXcds;
  size_t pos = 0;
  for (int x = 0; x < kXcds; ++x) {
    while (pos < other_items.size() &&
           (x == kXcds - 1 || load[x] + other_items[pos].cost <= target)) {
      q[x].push_back(other_items[pos].w);
      load[x] += other_items[pos].cost;
      ++pos;
    }
  }
  // longest first inside each queue, by length class of 16 key tiles
  // (stable: items of one class keep their locality order; sorting by the
  // exact length would move the 11-tile paired visual items away from their
  // 10-tile neighbours and cost the L2 their shared key/value tiles)
  for (int x = 0; x < kXcds; ++x) {
    std::stable_sort(q[x].begin(), q[x].end(),
                     [](const WorkItem& a, const WorkItem& b) {
                       return (a.kb_end - a.kb_begin + 15) / 16 >
                              (b.kb_end - b.kb_begin + 15) / 16;
                     });
  }
  size_t rounds = 0;
  for (auto& v : q) rounds = std::max(rounds, v.size());
  P.items.reserve(rounds * kXcds);
  for (size_t r = 0; r < rounds; ++r)
    for (int x = 0; x < kXcds; ++x) {
      if (r < q[x].size()) {
        P.items.push_back(q[x][r]);
      } else {
        WorkItem pad{-1, 0, 0, 0, 0, -1, 0, 0, -1, -1};
        P.items.push_back(pad);
      }
    }
  // drop trailing padding
  while (!P.items.empty() && P.items.back().qblock < 0) P.items.pop_back();
  for (WorkItem& w : P.items) {
    if (w.qblock < 0) continue;
    const BlockDesc& a = P.blocks[w.qblock];
    const BlockDesc& b = P.blocks[w.qblock2 >= 0 ? w.qblock2 : w.qblock];
    w.q0start = a.start;
    w.q0len = a.len;
    w.q1start = b.start;
    w.q1len = b.len;
    w.k0start = 0;
    w.k0len = 1;
    w.k1start = 0;
    w.k1len = 0;
    const std::vector<BlockDesc>& kd =
        w.qblock2 >= 0 ? P.ptile_desc : P.col_desc;
    if (w.kb_end > w.kb_begin) {
      w.k0start = kd[w.kb_begin].start;
      w.k0len = kd[w.kb_begin].len;
    }
    if (w.kb_end > w.kb_begin + 1) {
      w.k1start = kd[w.kb_begin + 1].start;
      w.k1len = kd[w.kb_begin + 1].len;
    }
  }
  for (const WorkItem& w : P.items)
    P.max_item_candidates =
        std::max(P.max_item_candidates, w.kb_end - w.kb_begin);
  return "";
}

}  // namespace evisel

// Internal runtime structures of libwf: workspace carve-up, parameter views and
// kernel launchers.  Not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/wf.h"
#include "wf_common.h"
#include "wf_kernels.h"

namespace wf {

// Offsets (in elements of the storage type) of one decoder block's parameters
// inside the weight region.  q/k/v are stored concatenated ([3d, d] and [3d]
// bias with a zero key bias), as are the cross-attention k/v ([2d, d], [2d]).
struct BlockW {
  size_t ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o;
  size_t ln2_g, ln2_b, w_q2, b_q2, w_kv2, b_kv2, w_o2, b_o2;
  size_t ln3_g, ln3_b, w_fc1, b_fc1, w_fc2, b_fc2;
  // fp32 offsets (in the LayerNorm column-sum region) of c then e for the products
  // with a LayerNorm folded in: q|k|v (3 d each), W'_q (d), W_1 (d_ff)
  size_t c_qkv, c_q2, c_fc1;
};

struct Layout {
  // byte offsets into the workspace
  size_t state, page_table, rope, status, aux, weights, xkv, skv, hkv;
  size_t a_d16, a_d32, a_f16, a_tap16, h, qkv, hp, kvh, hv, hi, tok, g, gmax, draft, lasth, logits, dlogits, part;
  size_t hm, hs, tmax, tsum, dmax, dsum, sst, spart;  // sampling: normalisers and draw partials
  size_t xpart;   // chunked cross-attention: partial records
  size_t lncd;    // LayerNorm column sums of the folded products (batch 1, bf16)
  size_t stamps;  // launch timing slots (profiling)
  size_t total;
  // element offsets inside the weight region
  size_t tok_emb, pos_emb, lnf_g, lnf_b, hproj_w, hproj_b, mask, dlnf_g, dlnf_b;
  // fp32 offsets (column-sum region) of the heads' c then e: the final LayerNorm of
  // the target (lnf) and of the drafter (dlnf) folded into the vocabulary product
  size_t c_head, c_dhead;
  std::vector<BlockW> tb, db;
  size_t weight_elems;
  int pages_per_slot, head_blocks;
  int nsplit_op;  // bf16 terms of a matrix operand value (3: rows, batch 1; 2: planes, several slots; fp32: 1)
  int mt16, mt32; // 16-row / 32-row tiles held by an operand buffer
  size_t stage_bytes;  // raw-matrix staging at init (inside the cross K/V region)
  int fc2_split;       // k-splits of the second MLP product (0: not split)
};

struct Handle;

constexpr int kFc2SplitBatch = 4;  // k-splits of the second MLP product with several slots
constexpr int kResidSplit = 4;     // k-splits of the attention output products for small multi-slot batches

struct GraphKey {
  int slot0, n, k_max;
  const void *ovr, *out, *nout, *nacc, *done;
  bool prof;  // captured with event records around every launch
  bool operator<(const GraphKey& o) const {
    return std::tie(slot0, n, k_max, ovr, out, nout, nacc, done, prof) <
           std::tie(o.slot0, o.n, o.k_max, o.ovr, o.out, o.nout, o.nacc, o.done, o.prof);
  }
};

struct ProfRec {
  const char* tag;
  double bytes;
  int slot;  // timing slot in the stamp buffer
};
struct ProfAgg {
  double ms = 0;       // end of the previous launch's last wave to the end of this one's
  double exec_ms = 0;  // first-wave start to last-wave end
  double bytes = 0;
  long n = 0;
};

struct Handle {
  wf_config cfg;
  Layout lay;
  char* ws;
  size_t ws_bytes;
  float temperature = 0.f;
  float inv_t = 0.f;  // fp32(1 / temperature) when sampling
  uint64_t seed = 0;
  const uint8_t* suppress = nullptr;
  bool debug = false;
  std::string err;
  std::vector<int> live;  // host mirror: slot prefilled
  std::map<GraphKey, hipGraphExec_t> graphs;
  bool prof = false;       // time launches (eager calls and profiled graph replays)
  bool capturing = false;  // inside graph capture
  int nstamp = 0;          // timing slots handed out in the current call or capture
  std::vector<ProfRec> prof_recs;                        // launches of the current eager call
  std::vector<ProfRec> cap_recs;                         // launches of the graph being captured
  std::map<GraphKey, std::vector<ProfRec>> graph_recs;  // launches of each profiled graph
  std::map<std::string, ProfAgg> prof_acc;              // durations per launch class
  double wall_khz = 0;                                   // device wall-clock rate
  int device = 0;          // device that was current when the handle was created
  // Non-null only inside a wf_step_noalloc call: the per-call buffers (the byte
  // range [lay.a_d16, lay.lncd) of the workspace: operands, activation rows,
  // partial sums, head partials, logits) then live at this device address, the
  // library's static scratch array, instead of the workspace.
  char* scratch = nullptr;

  template <typename T>
  T* at(size_t off) const {
    if (scratch && off >= lay.a_d16 && off < lay.lncd) return reinterpret_cast<T*>(scratch + (off - lay.a_d16));
    return reinterpret_cast<T*>(ws + off);
  }
  // bytes of the per-call buffers (what wf_step_noalloc places in the static scratch)
  size_t transient_bytes() const { return lay.lncd - lay.a_d16; }
};

int compute_layout(const wf_config& c, Layout& L);

}  // namespace wf

// Internal plan structure shared by the planner (plan.cpp) and the band
// executor (exec.cpp). Host memory only.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "lrcnn.h"

namespace lrcnn {

struct Shape {
  int h, w, c;
};

// Rows of one node in one band: [a, b) computed and owned by the band,
// [lo, hi) held in the band's window buffer (lo <= a, b == hi).
struct Rows {
  int a, b, lo, hi;
};

// Byte offsets of every buffer inside one workspace.
struct Layout {
  size_t total = 0;
  size_t arena = 0, arena_bytes = 0;  // backward arena (idle during the forward pass)
  size_t ubase = 0;              // start of the region FP and BP share
  std::vector<size_t> win;       // per node: feature-map window ([B][cap][W][C])
  std::vector<int> win_cap;      // rows of each window
  std::vector<size_t> argmax;    // per MAXPOOL node: uint8 argmax of own rows
  std::vector<int> argmax_cap;
  std::vector<size_t> delta;     // per node: float32 error window
  std::vector<size_t> carry;     // per node: float32 error carried to band r-1
  // per node whose consumer's backward launch writes its carried rows: a
  // second carry buffer; bands of odd index write (and the band below
  // reads) this one, so that launch never writes the buffer it reads the
  // rows carried in from (0: one buffer)
  std::vector<size_t> carry2;
  std::vector<int> carry_cap;
  std::vector<std::vector<size_t>> strip;  // [band][node]: shared rows kept
  size_t part = 0, part_bytes = 0;  // split-K partial sums (forward, input gradient)
  // per conv node, in the BP arena: error operand (storage dtype) and
  // weight-gradient partial sums
  std::vector<size_t> dc, wpart, wpart_bytes;
  // input with a channel count that is not a multiple of one 16-byte vector:
  // a channel-padded copy of the rows a first-layer weight gradient reads,
  // and that gradient accumulated in padded form [C_out][taps][cpad]
  int cpad = 0, xpad_cap = 0;
  size_t xpad = 0;
  std::vector<size_t> dwpad;
  size_t dxacc = 0, dxacc_bytes = 0;  // RECOMPUTE: float32 dX accumulator
  // per conv node: the most output rows one forward launch may cover, so
  // that its split-K partial sums fit `part_bytes` (0: no limit)
  std::vector<int> fchunk;
  size_t strip_bytes = 0, cache_bytes = 0, delta_bytes = 0, carry_bytes = 0;
  // forward windows packed by lifetime (when the forward partition is
  // coarser than the backward one); they share memory with the buffers that
  // only the backward pass uses
  bool fp_packed = false;
  std::vector<size_t> fwin;
  std::vector<int> fwin_cap;
  size_t fwin_bytes = 0;
};

// Fusions of a schedule (decided from that schedule's own rows, so the
// layer-wise baseline does not depend on the row partition):
//  add[u]: the ADD node whose backward writes conv u's error operand
//          directly (a conv without ReLU whose only consumer is that add
//          and that carries no rows between backward bands), else 0
//  fwd[u]: the ADD node whose forward conv u's epilogue computes (the add's
//          later input, fused in its backward, same rows in every band and
//          whole 16-byte channel vectors), else 0
//  act[u]: (CARRY / layer-wise) conv u's only consumer, a conv or max-pool
//          v, whose backward launch forms u's error operand and carry
//          directly (when that launch initializes u's whole error window);
//          u's error operand then lives from v's backward step
struct Fuse {
  std::vector<int> add, fwd, act;
};

struct Plan {
  std::vector<lrcnn_node> nodes;
  lrcnn_config cfg{};
  int n = 0, nb = 0, es = 4;  // node count, backward band count, element size
  int nb_fp = 0, refine = 1;  // forward band count, backward bands per forward band
  std::vector<Shape> shp;
  std::vector<std::vector<int>> cons;  // consumers of every node
  std::vector<int> bounds;             // backward band bounds (input or output rows)
  std::vector<int> bounds_fp;          // forward band bounds
  std::vector<std::vector<Rows>> rows; // [backward band][node]
  std::vector<std::vector<Rows>> rows_fp;  // [forward band][node]
  std::vector<std::vector<int>> tail;  // CARRY: [backward band][node] first kept row
  Fuse fz;     // fusions of the row-centric schedule
  Fuse fz_lw;  // fusions of the layer-wise schedule
  // per conv node: the split-K count of every forward launch (row-centric
  // bands, recompute and layer-wise alike), so each output element sums
  // its K products in the same order in every schedule (0: not a conv)
  std::vector<int> fsplit;
  // hybrid parts: the whole plan's counts for their nodes (so the hybrid's
  // forward equals the whole plan's layer-wise forward bit for bit)
  std::vector<int> fsplit_fixed;
  Layout rc;                           // row-centric workspace
  Layout lw;                           // layer-wise workspace
  double tau = 0, flops_rows = 0;
  int64_t shared_rows = 0, halo_rows = 0;
  // state for the FP -> BP hand-over of CARRY mode
  const void *fwd_workspace = nullptr;
  uint64_t fwd_epoch = 0;
  bool last_band_kept = false;  // FP left the last band's maps in place
  // side stream and two events of the backward, created by the executor on
  // first use for the device current at that call (opaque HIP handles)
  void *side_stream = nullptr, *ev_act = nullptr, *ev_wg = nullptr;
  // forward pass pipelined over bands: per node, an event after each of two
  // bands' steps (band parity), and one to fork the side stream
  std::vector<void *> ev_fp;
  void *ev_fork = nullptr;
  int side_dev = -1;
  // hybrid depth: nodes < hyb row-centric (sub-plan `row`, nodes 0..hyb-1),
  // nodes >= hyb layer-wise (sub-plan `col`, re-indexed from the checkpoint
  // node hyb-1 as its input). Workspace: the row part's layout; the column
  // part's layer-wise layout overlays the row part's shared FP/BP region
  // (idle between the two parts); then the checkpoint map (storage dtype)
  // and its float32 error.
  int hyb = 0;
  Plan *row = nullptr, *col = nullptr;
  size_t h_col = 0, h_ck = 0, h_dck = 0, h_total = 0;
  bool no_keep = false;      // FP must not leave its last band for BP
  bool dy_f32 = false;       // dL/dy is float32 (a checkpoint's error)
  bool lw_keep_out = false;  // layer-wise layout keeps the output node's map
  ~Plan() {
    delete row;
    delete col;
  }

  size_t elems(int v, int rows_) const {
    return (size_t)cfg.batch * rows_ * shp[v].w * shp[v].c;
  }
};

// Releases the executor's side stream and events of a plan (exec.cpp).
void release_side(Plan &P);

// planning on the calling thread forms every error operand by its own
// activation-backward pass (test hook)
extern thread_local bool g_no_act_fusion;

}  // namespace lrcnn

// Thread-local error reporting shared by all translation units.
int lrcnn_fail(int code, const std::string &msg);

// Host planner: validates one micro-batch's metadata and lays out the device
// workspace and tape.  Pure C++ (no HIP), so every check runs before any launch.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

namespace mpipe {

struct Cfg {
  int in_chans = 3, patch = 14, tpatch = 1, hidden = 0, layers = 0, heads = 0, mlp = 0,
      merge = 2, llm = 0, dtype = 1;
  float eps = 1e-6f, theta = 10000.f;
  // derived
  int d = 0;        // head dim
  int kpe = 0;      // patch vector length C*T*P*P
  int kp = 0;       // kpe rounded up to the GEMM K step (64)
  int esz = 2;      // bytes per activation element
};

// Returns "" when cfg is supported, else the reason.
std::string check_cfg(const Cfg& c);
void derive_cfg(Cfg& c);

struct ParamEntry {
  std::string name;
  int64_t off, rows, cols;
};
std::vector<ParamEntry> param_table(const Cfg& c);

// indices into param_table
constexpr int P_PE_W = 0, P_PE_B = 1, P_BLK0 = 2, P_PER_BLK = 12;
enum { B_LN1G, B_LN1B, B_QKVW, B_QKVB, B_PROJW, B_PROJB, B_LN2G, B_LN2B, B_FC1W, B_FC1B,
       B_FC2W, B_FC2B };
enum { M_LNG, M_LNB, M_FC1W, M_FC1B, M_FC2W, M_FC2B };
inline int blk_param(const Cfg& c, int layer, int which) {
  (void)c;
  return P_BLK0 + P_PER_BLK * layer + which;
}
inline int merger_param(const Cfg& c, int which) { return P_BLK0 + P_PER_BLK * c.layers + which; }

// Byte offsets of one layer's activations (in the tape when trainable, in the
// workspace -- shared by all layers -- when frozen).
struct ActSet {
  size_t hin, hmid, hout;        // fp32 [N][h] residual stream: in, after attention, out
  size_t a, b;                   // LN1 / LN2 outputs [N][h]
  size_t mean1, rstd1, mean2, rstd2;  // fp32 [N]
  size_t qkv;                    // [N][3h] (q, k after rotary)
  size_t o;                      // attention output [N][h]
  size_t lse;                    // fp32 [heads][N]
  size_t u;                      // fc1 pre-activation [N][m] (trainable only)
  size_t g;                      // GELU output [N][m]
};
struct MergerSet {
  size_t hfin;                   // fp32 [N][h] (the last layer's hout)
  size_t z, meanz, rstdz;        // LN output [N][h] (= [Tm][4h]), fp32 stats
  size_t um, gm;                 // [Tm][4h] pre-activation / GELU output
};

// Largest grid side (in patches) an item may have: positions are packed as y << 16 | x,
// so each coordinate must fit in 15 bits.
constexpr int kMaxGridSide = 32768;

// Upper bound of the partial-sum rows of the deterministic column reductions (LayerNorm
// backward blocks, column-sum chunks); the workspace holds this many rows per reduction.
constexpr int64_t kPartialRowsMax = 1024;

struct GemmSplit {
  int splits = 1;
  int kps = 0;
};
GemmSplit choose_split(int64_t M, int64_t N, int64_t K);

// Trainability modes (the C ABI's mpipe_train_mode): nothing, everything, or only the
// merger trainable.
enum { MODE_FROZEN = 0, MODE_TRAINED = 1, MODE_MERGER = 2 };

// A byte range [off, off + bytes) of the workspace or the tape.
struct Region {
  size_t off, bytes;
};

struct Plan {
  int64_t N = 0, Tm = 0;
  int n_items = 0, n_seg = 0;
  int mode = MODE_FROZEN;
  bool trainable = false;          // mode == MODE_TRAINED: every layer records a tape
  int64_t sum_len2 = 0;          // sum over segments of len^2 (attention FLOPs)
  // host metadata, uploaded into the workspace head
  std::vector<int32_t> pos;        // N: y << 16 | x (y, x < kMaxGridSide)
  std::vector<int32_t> q_work;     // 4 ints per query tile (start, seg start, seg end, 0)
  std::vector<int32_t> k_work;     // 4 ints per key tile
  std::vector<float> rope_tab;     // (cos, sin) of p * theta^(-4k/d), [positions][d/4]
  size_t meta_bytes = 0;
  // workspace layout
  size_t ws_pos = 0, ws_qwork = 0, ws_kwork = 0, ws_rope = 0;
  size_t ws_xp = 0, ws_wpe = 0;
  size_t ws_wt = 0;                // the forward's transposed weights, one layer at a time
  ActSet ws_act{};                 // frozen forward activations
  MergerSet ws_mrg{};
  size_t ws_dh = 0, ws_dht = 0, ws_dhm = 0, ws_dhmt = 0, ws_dxln = 0, ws_du = 0, ws_do = 0,
         ws_delta = 0, ws_dqkv = 0, ws_dqkv2 = 0, ws_part = 0, ws_cpart = 0, ws_dwpart = 0,
         ws_gpart = 0;
  size_t ws_bytes = 0;
  std::vector<Region> ws_regions;   // every range a kernel may write, in layout order
  // tape layout: every layer and the merger (MODE_TRAINED), the merger only (MODE_MERGER)
  std::vector<ActSet> tape_act;
  MergerSet tape_mrg{};
  size_t tape_bytes = 0;
  std::vector<Region> tape_regions;
};

// W (FLOPs) and D (algorithmic HBM bytes) of one micro-batch's forward and backward
// slabs in the plan's trainability mode (owner.cpp).
struct SlabCost {
  double fwd_flops = 0, fwd_bytes = 0, bwd_flops = 0, bwd_bytes = 0;
};
SlabCost encoder_slab_cost(const Cfg& c, const Plan& P);

// (cos, sin) table of the rotary angles p * theta^(-4k/d) for p < positions, k < d/4.
std::vector<float> rope_table(const Cfg& c, int positions);

// Validate metadata and build the plan for a trainability mode (MODE_*).  Returns 0 or
// a negative mpipe_status; `err` receives the reason.
int build_plan(const Cfg& c, const int32_t* cu, int n_seg, const int32_t* thw, int n_items,
               int mode, Plan& p, std::string& err);

}  // namespace mpipe

// Internal declarations shared by the TRA library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "tra.h"

namespace tra {

// Packed token coordinate of a tile-major position: y in bits 0-9, x in bits
// 10-19, f in bits 20-25 (the plan limits W, H <= 1023 and F <= 64).
__host__ __device__ inline int32_t pack_coord(int f, int x, int y) {
  return (f << 20) | (x << 10) | y;
}
__host__ __device__ inline int coord_f(int32_t c) { return c >> 20; }
__host__ __device__ inline int coord_x(int32_t c) { return (c >> 10) & 1023; }
__host__ __device__ inline int coord_y(int32_t c) { return c & 1023; }

// per block: f_min f_max x_min x_max y_min y_max n_video r_min r_max n_text
constexpr int kBlockInfo = 10;
constexpr int kKeyInfo = 128;  // ints per key block in the key-info table
constexpr int kKeyFeat = 8;    // f16 values per key in the key-feature table (2-D token mask)
constexpr int kMaxFrames = 64;
constexpr int kMaxBlocks = 4096;
constexpr int kSortChunk = 256;
constexpr int kRowCounters = 128;  // ints of the attention row-queue counters

// Host-side tables of one shape (plan.cpp).
struct HostTables {
  int32_t N = 0, S = 0, NB = 0, n_cap = 0;  // video tokens, all tokens, blocks of the layout
  int32_t P = 0;                // positions of the block layout's order (S packed, NB * b tiles)
  std::vector<int32_t> perm;    // [P] position -> token index (text: N + t), -1 = padding
  std::vector<int32_t> perm_attn;  // tile-aligned layout only: the packed order [S]
  std::vector<int32_t> coord;   // [P] packed (f, x, y) of a video position, 0 otherwise
  std::vector<int32_t> thr;     // [(n_cap + 1) * F] 2-D squared thresholds
  std::vector<int32_t> thr1;    // [(n_cap + 1) * F] 1-D thresholds
  std::vector<int32_t> blocks;  // [NB * kBlockInfo]
  std::vector<int32_t> kinfo;   // [(NB + 1) * kKeyInfo]
  std::vector<uint16_t> kfeat;  // 2-D distance: [NB][2][block][4] f16 bit patterns (components 4h..4h+3 at h)
};

// f16 bit pattern of an integer v with |v| <= 2048 (exact).
uint16_t f16_bits_of_int(int v);

// Phi^{-1}(p) of the standard normal in fp64, by bisection on Phi.
double normal_quantile(double p);

// Validates the config; on failure returns the status and fills `why`.
tra_status validate_config(const tra_config* cfg, std::string* why);
void build_host_tables(const tra_config& cfg, HostTables* t, bool with_perm_coord,
                       bool with_thr, bool with_thr1, bool with_blocks, bool with_kinfo = false);

}  // namespace tra

struct tra_plan_s {
  tra_config cfg;
  int device = 0;
  int32_t N = 0;   // video tokens F*H*W
  int32_t S = 0;   // all tokens (video then text): the row length of every tensor
  // Block layout (mask, block-sparse and token-level calls): NB blocks per
  // head, rows = batch * heads * NB query-block rows, n_pad = NB * block
  // positions; d_perm [n_pad]: position -> token, -1 at padding (the packed
  // layout's positions past S, a clipped tile's tail); d_coord [n_pad];
  // d_bcount [NB]: tokens of each block (they fill its first positions).
  int32_t NB = 0, n_cap = 0, rows = 0;
  double z_tau = 0.0;  // Phi^{-1}(tau), lognormal budget mapping
  int32_t* d_perm = nullptr;
  int32_t* d_coord = nullptr;
  int32_t* d_bcount = nullptr;
  // Layout of the calls defined over tokens (entropy, dense): always the
  // packed order.  Equal to the block layout's fields for packed plans (the
  // same device table); for tile-aligned plans a table of its own.
  int32_t NBa = 0, rowsa = 0, n_pada = 0;
  int32_t* d_perma = nullptr;
  int32_t* d_thr = nullptr;
  int32_t* d_thr1 = nullptr;  // 1-D thresholds (TRA_DIST_1D plans only)
  int32_t* d_blocks = nullptr;
  // C(n) of every candidate radius over one octant of the grid (App. C.1's
  // lookup table), or NULL above kCountTableMaxBytes; then d_cap_count holds
  // C(n_cap) per video position (raster) and the other counts run on the fly
  int32_t* d_ctab = nullptr;
  int32_t* d_cap_count = nullptr;
  // Per-call device memory.  The pointers below marked "call workspace" are
  // NULL in a stored plan, which no call writes; each call works on a copy of
  // the plan with them pointing into the caller's workspace buffer.
  int32_t* d_sort_ws = nullptr;  // call workspace: counting-sort histograms of the row order
  int64_t sort_ws_elems = 0;
  int32_t sort_chunks = 0;
  // bf16 plans, call workspace: K and V gathered into tile-major order,
  // [batch*heads][NB*block][d] (V transposed in 64-key tiles), rows past S
  // zero-filled, so the attention loop addresses tiles affinely.
  int32_t n_pad = 0;
  uint16_t* d_kt = nullptr;
  uint16_t* d_vt = nullptr;
  // bf16 plans: per key block, 128 distance words (2-D: x | y << 16; 1-D: the
  // raster index) with a second-frame flag and a text flag, [NB + 1][128],
  // the key side of the token mask inside a tile.
  int32_t* d_kinfo = nullptr;
  // bf16 plans with the 2-D distance: per key, 8 f16 integers b with
  // a_i . b_j = T_i(frame of j) - D_ij for the query vector a_i the token
  // kernel forms per tile, [NB][2][128][4] (see build_host_tables).
  uint16_t* d_kfeat = nullptr;
  int32_t thr_max = 0;  // largest entry of the plan's threshold table
  // bf16 plans, call workspace: row-queue counters of the persistent attention
  // kernel (kRowCounters ints, reset by each call on its stream); the CU count
  int32_t* d_row_ctr = nullptr;
  int32_t n_cu = 0;
  // bf16 plans, call workspace: work units of block-sparse calls (rows cut into pieces of at
  // most L list entries) and the pieces' partial results: units [units_cap]
  // int4, split rows [splits_cap] int4, header {units, split rows, L, 0, nine
  // segment starts of the per-XCD queues} (kUnitHdrInts ints), partial
  // outputs [slots_cap][128][d] fp32 and statistics [slots_cap][3][128] fp32
  // (running max, rounded and fp32 sums), for at most split_wg_cap workgroups;
  // the capacities are the plan's, fixed at creation.
  int32_t split_wg_cap = 0, units_cap = 0, splits_cap = 0, slots_cap = 0;
  int32_t* d_units = nullptr;
  int32_t* d_splits = nullptr;
  int32_t* d_unit_hdr = nullptr;
  float* d_part = nullptr;
  float* d_pstats = nullptr;
};

namespace tra {

// ----------------------------------------------------------- kernel launchers
// Each returns hipSuccess or the launch error.  All run on `stream`.

// Attention family.  mode flags select the variant.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  float* entropy;
  const int32_t* cnt;    // sparse only
  const int32_t* cols;   // sparse only
  const int32_t* order;  // sparse only, may be null
  bool sparse;
  const int32_t* radius_sq = nullptr;  // token-level attention (sparse) only
  // kernel timing: recorded on the call's stream around the attention kernel
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
};
hipError_t launch_attention_bf16(const tra_plan_s& p, const AttnArgs& a, hipStream_t s);
// Largest grid of the block-sparse attention kernel on this plan's device, and
// the work-unit table capacities for that grid.
int k64_sparse_grid_cap(const tra_plan_s& p);
void split_capacities(int grid_cap, int rows, int NB, int head_dim, int* units_cap, int* splits_cap,
                      int* slots_cap);
constexpr int kUnitHdrInts = 16;  // header of the work-unit tables
hipError_t launch_attention_f32(const tra_plan_s& p, const AttnArgs& a, hipStream_t s);

hipError_t launch_budget_radius(const tra_plan_s& p, const float* entropy, int32_t* budget,
                                int32_t* radius_sq, hipStream_t s);
// Fills the plan's per-position table of C(n_cap) (once, at plan creation).
hipError_t fill_cap_counts(const tra_plan_s& p, int32_t* out, hipStream_t s);
// The count table of App. C.1 over one octant of the grid: its size, and its
// fill (disk_tmp: ceil(H/2) ceil(W/2) (n_cap + 1) ints of scratch).
constexpr size_t kCountTableMaxBytes = (size_t)1 << 30;
size_t count_table_bytes(const tra_plan_s& p);
hipError_t fill_count_table(const tra_plan_s& p, int32_t* ctab, int32_t* disk_tmp, hipStream_t s);

hipError_t launch_block_mask(const tra_plan_s& p, const int32_t* radius_sq, uint8_t* mask,
                             int32_t* cnt, int32_t* cols, hipStream_t s);

hipError_t launch_row_order(const tra_plan_s& p, const int32_t* cnt, int32_t* order,
                            hipStream_t s);

// The no-allocation variant: the same order with its counting-sort workspace
// in the library's per-device scratch array of kNoAllocScratchInts ints.
constexpr int64_t kNoAllocScratchInts = (int64_t)1 << 20;  // 4 MiB
// Device address of that array on `device` (the current device), resolved once
// per device and kept.
hipError_t resolve_noalloc_scratch(int device, int32_t** out);
hipError_t launch_row_order_noalloc(const tra_plan_s& p, const int32_t* cnt, int32_t* order,
                                    hipStream_t s);

}  // namespace tra

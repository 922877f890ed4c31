// C ABI entry points of the TRA library: argument checks, plan lifetime,
// dispatch to the kernel launchers.  No exception leaves this file.
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "tra_internal.h"

namespace {

thread_local std::string g_last_error;

tra_status fail(tra_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

tra_status ok() {
  g_last_error.clear();
  return TRA_OK;
}

tra_status hip_fail(hipError_t e, const char* what) {
  return fail(TRA_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// The plan's device must be current: kernels index the plan's tables.
tra_status check_plan(tra_plan p) {
  if (!p) return fail(TRA_ERR_INVALID_ARG, "plan is NULL");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != p->device)
    return fail(TRA_ERR_INVALID_ARG, "current device differs from the plan's device");
  return TRA_OK;
}

tra_status check_tensor(const void* ptr, const char* name, bool nullable = false) {
  if (!ptr) {
    if (nullable) return TRA_OK;
    return fail(TRA_ERR_INVALID_ARG, std::string(name) + " is NULL");
  }
  if (!aligned16(ptr)) return fail(TRA_ERR_INVALID_ARG, std::string(name) + " is not 16-byte aligned");
  return TRA_OK;
}

tra_status check_aligned4(const void* ptr, const char* name, bool nullable) {
  if (!ptr) {
    if (nullable) return TRA_OK;
    return fail(TRA_ERR_INVALID_ARG, std::string(name) + " is NULL");
  }
  if (((uintptr_t)ptr & 3u) != 0) return fail(TRA_ERR_INVALID_ARG, std::string(name) + " is not 4-byte aligned");
  return TRA_OK;
}

#define TRA_TRY(expr)                   \
  do {                                  \
    tra_status _s = (expr);             \
    if (_s != TRA_OK) return _s;        \
  } while (0)

tra_status launch_result(hipError_t e, const char* what) {
  if (e != hipSuccess) return hip_fail(e, what);
  return ok();
}

// ----------------------------------------------------------- call workspace
// Device memory a call writes besides its outputs, carved from the caller's
// workspace buffer (each piece 256-byte aligned).  The plan itself holds only
// tables that no call writes.
constexpr size_t kWsAlign = 256;

struct WsLayout {
  size_t kt = 0, vt = 0, ctr = 0, units = 0, splits = 0, hdr = 0, part = 0, pstats = 0, sort = 0;
  size_t total = 0;
};

WsLayout ws_layout(const tra_plan_s& p, int call) {
  WsLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + kWsAlign - 1) / kWsAlign * kWsAlign;
    return at;
  };
  if (call == TRA_CALL_BLOCK_MASK) {
    L.sort = take((size_t)p.sort_ws_elems * sizeof(int32_t));
  } else if (p.cfg.dtype == TRA_BF16) {
    const size_t kv =
        (size_t)p.cfg.batch * p.cfg.heads * std::max(p.n_pad, p.n_pada) * p.cfg.head_dim * sizeof(uint16_t);
    L.kt = take(kv);
    L.vt = take(kv);
    L.ctr = take(tra::kRowCounters * sizeof(int32_t));
    if (call == TRA_CALL_SPARSE) {
      L.units = take((size_t)p.units_cap * 4 * sizeof(int32_t));
      L.splits = take((size_t)p.splits_cap * 4 * sizeof(int32_t));
      L.hdr = take(tra::kUnitHdrInts * sizeof(int32_t));
      L.part = take((size_t)p.slots_cap * 128 * p.cfg.head_dim * sizeof(float));
      L.pstats = take((size_t)p.slots_cap * 3 * 128 * sizeof(float));
    }
  }
  L.total = off;
  return L;
}

// Checks the caller's workspace for `call` and returns, in *out, a copy of the
// plan whose per-call pointers address it.  `needed` is false where the call
// writes no workspace (then the buffer may be NULL).
tra_status bind_workspace(tra_plan p, int call, bool needed, void* ws, size_t ws_bytes, tra_plan_s* out) {
  *out = *p;
  const WsLayout L = ws_layout(*p, call);
  if (!needed || L.total == 0) return TRA_OK;
  if (!ws)
    return fail(TRA_ERR_INVALID_ARG, "workspace is NULL; this call needs " + std::to_string(L.total) +
                                         " bytes (tra_workspace_size)");
  if (((uintptr_t)ws & (kWsAlign - 1)) != 0)
    return fail(TRA_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
  if (ws_bytes < L.total)
    return fail(TRA_ERR_INVALID_ARG, "workspace holds " + std::to_string(ws_bytes) + " bytes; this call needs " +
                                         std::to_string(L.total) + " (tra_workspace_size)");
  uint8_t* b = (uint8_t*)ws;
  if (call == TRA_CALL_BLOCK_MASK) {
    out->d_sort_ws = (int32_t*)(b + L.sort);
    return TRA_OK;
  }
  out->d_kt = (uint16_t*)(b + L.kt);
  out->d_vt = (uint16_t*)(b + L.vt);
  out->d_row_ctr = (int32_t*)(b + L.ctr);
  if (call == TRA_CALL_SPARSE) {
    out->d_units = (int32_t*)(b + L.units);
    out->d_splits = (int32_t*)(b + L.splits);
    out->d_unit_hdr = (int32_t*)(b + L.hdr);
    out->d_part = (float*)(b + L.part);
    out->d_pstats = (float*)(b + L.pstats);
  }
  return TRA_OK;
}

}  // namespace

extern "C" {

const char* tra_last_error(void) { return g_last_error.c_str(); }

const char* tra_version(void) { return "tra-mi355x 0.1 (gfx950)"; }

tra_status tra_plan_host_tables(const tra_config* cfg, int32_t* perm, int32_t* thr,
                                int32_t* thr1, int32_t* blocks, int32_t* n_cap_out) {
  try {
    std::string why;
    tra_status s = tra::validate_config(cfg, &why);
    if (s != TRA_OK) return fail(s, why);
    tra::HostTables t;
    tra::build_host_tables(*cfg, &t, perm != nullptr, thr != nullptr, thr1 != nullptr,
                           blocks != nullptr);
    if (perm) std::memcpy(perm, t.perm.data(), t.perm.size() * sizeof(int32_t));  // P entries
    if (thr) std::memcpy(thr, t.thr.data(), t.thr.size() * sizeof(int32_t));
    if (thr1) std::memcpy(thr1, t.thr1.data(), t.thr1.size() * sizeof(int32_t));
    if (blocks) std::memcpy(blocks, t.blocks.data(), t.blocks.size() * sizeof(int32_t));
    if (n_cap_out) *n_cap_out = t.n_cap;
    return ok();
  } catch (const std::bad_alloc&) {
    return fail(TRA_ERR_ALLOC, "host allocation failed");
  } catch (...) {
    return fail(TRA_ERR_INVALID_ARG, "unexpected error building host tables");
  }
}

tra_status tra_plan_destroy(tra_plan p) {
  if (!p) return ok();
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(p->device);
  if (p->d_perma != p->d_perm) (void)hipFree(p->d_perma);
  (void)hipFree(p->d_perm);
  (void)hipFree(p->d_coord);
  (void)hipFree(p->d_bcount);
  (void)hipFree(p->d_thr);
  (void)hipFree(p->d_thr1);
  (void)hipFree(p->d_blocks);
  (void)hipFree(p->d_cap_count);
  (void)hipFree(p->d_ctab);
  (void)hipFree(p->d_kinfo);
  (void)hipFree(p->d_kfeat);
  if (prev >= 0) (void)hipSetDevice(prev);
  delete p;
  return ok();
}

tra_status tra_plan_create(const tra_config* cfg, tra_plan* out) {
  if (!out) return fail(TRA_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  try {
    std::string why;
    tra_status s = tra::validate_config(cfg, &why);
    if (s != TRA_OK) return fail(s, why);

    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
      return fail(TRA_ERR_UNSUPPORTED, std::string("device is ") + prop.gcnArchName + ", not gfx950");

    tra::HostTables t;
    const bool one_d = cfg->distance == TRA_DIST_1D;
    tra::build_host_tables(*cfg, &t, true, true, one_d, true, cfg->dtype == TRA_BF16);

    tra_plan p = new tra_plan_s();
    p->cfg = *cfg;
    p->device = dev;
    p->n_cu = prop.multiProcessorCount;
    p->N = t.N;
    p->S = t.S;
    p->NB = t.NB;
    p->z_tau = tra::normal_quantile(cfg->tau);
    p->n_cap = t.n_cap;
    p->rows = cfg->batch * cfg->heads * t.NB;
    p->sort_chunks = (p->rows + tra::kSortChunk - 1) / tra::kSortChunk;
    // chunk histograms over keys 0..NB, plus one total slot
    p->sort_ws_elems = (int64_t)(t.NB + 1) * p->sort_chunks + 1;
    p->n_pad = t.NB * cfg->block;
    const bool tiles = cfg->block_layout == TRA_BLOCKS_TILES;
    p->NBa = tiles ? (t.S + cfg->block - 1) / cfg->block : t.NB;
    p->n_pada = p->NBa * cfg->block;
    p->rowsa = cfg->batch * cfg->heads * p->NBa;
    // the largest threshold: thr[n][0] = n, thr1[n][0] = floor(pi/2 n), at n = n_cap
    p->thr_max = one_d ? t.thr1[(size_t)t.n_cap * cfg->frames] : t.n_cap;

    auto upload = [&](int32_t** dst, const std::vector<int32_t>& src) -> hipError_t {
      hipError_t err = hipMalloc((void**)dst, src.size() * sizeof(int32_t));
      if (err != hipSuccess) return err;
      return hipMemcpy(*dst, src.data(), src.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    };
    // position tables padded to whole blocks: -1 (no token) / 0 past the order's end
    std::vector<int32_t> perm_pad = t.perm, coord_pad = t.coord, bcount(t.NB);
    perm_pad.resize(p->n_pad, -1);
    coord_pad.resize(p->n_pad, 0);
    for (int u = 0; u < t.NB; ++u)
      bcount[u] = t.blocks[(size_t)u * tra::kBlockInfo + 6] + t.blocks[(size_t)u * tra::kBlockInfo + 9];
    std::vector<int32_t> perma_pad = t.perm_attn;
    if (tiles) perma_pad.resize(p->n_pada, -1);
    if ((e = upload(&p->d_perm, perm_pad)) != hipSuccess ||
        (e = upload(&p->d_coord, coord_pad)) != hipSuccess ||
        (e = upload(&p->d_bcount, bcount)) != hipSuccess ||
        (tiles && (e = upload(&p->d_perma, perma_pad)) != hipSuccess) ||
        (e = upload(&p->d_thr, t.thr)) != hipSuccess ||
        (e = upload(&p->d_blocks, t.blocks)) != hipSuccess ||
        (one_d && (e = upload(&p->d_thr1, t.thr1)) != hipSuccess)) {
      tra_plan_destroy(p);
      return fail(TRA_ERR_ALLOC, std::string("plan table upload: ") + hipGetErrorString(e));
    }
    if (!tiles) p->d_perma = p->d_perm;
    // App. C.1's count table where it fits the size limit, else C(n_cap) per position
    const size_t ctab_bytes = tra::count_table_bytes(*p);
    if (ctab_bytes <= tra::kCountTableMaxBytes) {
      int32_t* disk_tmp = nullptr;
      const size_t disk_bytes = (size_t)((cfg->height + 1) / 2) * ((cfg->width + 1) / 2) * ((size_t)p->n_cap + 1) *
                                sizeof(int32_t);
      if ((e = hipMalloc((void**)&p->d_ctab, ctab_bytes)) != hipSuccess ||
          (e = hipMalloc((void**)&disk_tmp, disk_bytes)) != hipSuccess ||
          (e = tra::fill_count_table(*p, p->d_ctab, disk_tmp, nullptr)) != hipSuccess ||
          (e = hipStreamSynchronize(nullptr)) != hipSuccess) {
        (void)hipFree(disk_tmp);
        tra_plan_destroy(p);
        return fail(TRA_ERR_ALLOC, std::string("plan count table: ") + hipGetErrorString(e));
      }
      (void)hipFree(disk_tmp);
    } else if ((e = hipMalloc((void**)&p->d_cap_count, (size_t)std::max(p->N, 1) * sizeof(int32_t))) != hipSuccess ||
               (e = tra::fill_cap_counts(*p, p->d_cap_count, nullptr)) != hipSuccess ||
               (e = hipStreamSynchronize(nullptr)) != hipSuccess) {
      tra_plan_destroy(p);
      return fail(TRA_ERR_ALLOC, std::string("plan count table: ") + hipGetErrorString(e));
    }
    if (cfg->dtype == TRA_BF16) {
      if ((e = upload(&p->d_kinfo, t.kinfo)) != hipSuccess) {
        tra_plan_destroy(p);
        return fail(TRA_ERR_ALLOC, std::string("plan key-info table: ") + hipGetErrorString(e));
      }
      if (!t.kfeat.empty()) {
        const size_t bytes = t.kfeat.size() * sizeof(uint16_t);
        if ((e = hipMalloc((void**)&p->d_kfeat, bytes)) != hipSuccess ||
            (e = hipMemcpy(p->d_kfeat, t.kfeat.data(), bytes, hipMemcpyHostToDevice)) != hipSuccess) {
          tra_plan_destroy(p);
          return fail(TRA_ERR_ALLOC, std::string("plan key-feature table: ") + hipGetErrorString(e));
        }
      }
      p->split_wg_cap = tra::k64_sparse_grid_cap(*p);
      tra::split_capacities(p->split_wg_cap, p->rows, p->NB, cfg->head_dim, &p->units_cap, &p->splits_cap,
                           &p->slots_cap);
    }
    // the no-allocation entry point's scratch array on this device: its
    // address is resolved here, once per device, with the device current
    int32_t* scratch_ptr = nullptr;
    if ((e = tra::resolve_noalloc_scratch(dev, &scratch_ptr)) != hipSuccess) {
      tra_plan_destroy(p);
      return hip_fail(e, "hipGetSymbolAddress of the no-allocation scratch");
    }
    *out = p;
    return ok();
  } catch (const std::bad_alloc&) {
    return fail(TRA_ERR_ALLOC, "host allocation failed");
  } catch (...) {
    return fail(TRA_ERR_INVALID_ARG, "unexpected error creating plan");
  }
}

tra_status tra_workspace_size(tra_plan p, int32_t call, size_t* bytes) {
  if (!p) return fail(TRA_ERR_INVALID_ARG, "plan is NULL");
  if (!bytes) return fail(TRA_ERR_INVALID_ARG, "bytes is NULL");
  if (call < TRA_CALL_ENTROPY || call > TRA_CALL_DENSE)
    return fail(TRA_ERR_INVALID_ARG, "unknown call " + std::to_string(call));
  *bytes = ws_layout(*p, call).total;
  return ok();
}

tra_status tra_plan_dims(tra_plan p, int32_t* n_tokens, int32_t* n_blocks, int32_t* n_cap) {
  if (!p) return fail(TRA_ERR_INVALID_ARG, "plan is NULL");
  if (n_tokens) *n_tokens = p->S;
  if (n_blocks) *n_blocks = p->NB;
  if (n_cap) *n_cap = p->n_cap;
  return ok();
}

// Kernel timing state of the calling thread (tra_kernel_timing).  The events
// are not destroyed at thread exit (the runtime may be gone by then).
namespace {
struct KernelTiming {
  int call = -1, device = -1, used = 0;
  std::vector<hipEvent_t> start, stop;
  void release() {
    for (hipEvent_t e : start) (void)hipEventDestroy(e);
    for (hipEvent_t e : stop) (void)hipEventDestroy(e);
    start.clear();
    stop.clear();
    call = device = -1;
    used = 0;
  }
};
thread_local KernelTiming g_timing;
}  // namespace

tra_status tra_kernel_timing(int32_t call, int32_t n) {
  if (n < 0 || n > 4096) return fail(TRA_ERR_INVALID_ARG, "n must be in [0, 4096]");
  if (n > 0 && call != TRA_CALL_ENTROPY && call != TRA_CALL_SPARSE && call != TRA_CALL_TOKEN &&
      call != TRA_CALL_DENSE)
    return fail(TRA_ERR_INVALID_ARG, "call must be TRA_CALL_ENTROPY, _SPARSE, _TOKEN or _DENSE");
  g_timing.release();
  if (n == 0) return ok();
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "tra_kernel_timing: no device");
  for (int i = 0; i < n; ++i) {
    hipEvent_t a = nullptr, b = nullptr;
    if ((e = hipEventCreate(&a)) != hipSuccess || (e = hipEventCreate(&b)) != hipSuccess) {
      if (a) (void)hipEventDestroy(a);
      g_timing.release();
      return hip_fail(e, "tra_kernel_timing: event creation");
    }
    g_timing.start.push_back(a);
    g_timing.stop.push_back(b);
  }
  g_timing.call = call;
  g_timing.device = dev;
  return ok();
}

tra_status tra_kernel_times(float* ms, int32_t n, int32_t* got) {
  if (!got) return fail(TRA_ERR_INVALID_ARG, "got is NULL");
  if (n > 0 && !ms) return fail(TRA_ERR_INVALID_ARG, "ms is NULL");
  *got = g_timing.used;
  for (int i = 0; i < std::min<int>(n, g_timing.used); ++i) {
    hipError_t e = hipEventSynchronize(g_timing.stop[i]);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms[i], g_timing.start[i], g_timing.stop[i]);
    if (e != hipSuccess) return hip_fail(e, "tra_kernel_times");
  }
  return ok();
}

static tra_status run_attention(tra_plan p, int call, const tra::AttnArgs& a_in, void* ws, size_t ws_bytes,
                                void* stream, const char* what) {
  tra_plan_s bound;
  TRA_TRY(bind_workspace(p, call, true, ws, ws_bytes, &bound));
  tra::AttnArgs a = a_in;
  const bool timed = g_timing.call == call && g_timing.device == p->device &&
                     g_timing.used < (int)g_timing.start.size();
  if (timed) {
    a.ev_start = g_timing.start[g_timing.used];
    a.ev_stop = g_timing.stop[g_timing.used];
  }
  if (call == TRA_CALL_ENTROPY || call == TRA_CALL_DENSE) {
    // defined over tokens: run on the packed order whatever the block layout
    bound.NB = p->NBa;
    bound.n_pad = p->n_pada;
    bound.rows = p->rowsa;
    bound.d_perm = p->d_perma;
    bound.d_bcount = nullptr;  // packed: every block full but the last
  }
  hipError_t e = p->cfg.dtype == TRA_BF16
                     ? tra::launch_attention_bf16(bound, a, (hipStream_t)stream)
                     : tra::launch_attention_f32(bound, a, (hipStream_t)stream);
  if (timed && e == hipSuccess) ++g_timing.used;
  return launch_result(e, what);
}

tra_status tra_entropy(tra_plan p, const void* q, const void* k, const void* v, void* o,
                       float* entropy, void* workspace, size_t workspace_bytes, void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_tensor(q, "q"));
  TRA_TRY(check_tensor(k, "k"));
  TRA_TRY(check_tensor(v, "v", true));
  TRA_TRY(check_tensor(o, "o", true));
  TRA_TRY(check_aligned4(entropy, "entropy", false));
  if ((v == nullptr) != (o == nullptr))
    return fail(TRA_ERR_INVALID_ARG, "v and o must be both NULL or both non-NULL");
  tra::AttnArgs a{q, k, v, o, nullptr, entropy, nullptr, nullptr, nullptr, false};
  return run_attention(p, TRA_CALL_ENTROPY, a, workspace, workspace_bytes, stream, "tra_entropy launch");
}

tra_status tra_budget_radius(tra_plan p, const float* entropy, int32_t* budget,
                             int32_t* radius_sq, void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_aligned4(entropy, "entropy", false));
  TRA_TRY(check_aligned4(budget, "budget", true));
  TRA_TRY(check_aligned4(radius_sq, "radius_sq", false));
  return launch_result(tra::launch_budget_radius(*p, entropy, budget, radius_sq, (hipStream_t)stream),
                       "tra_budget_radius launch");
}

tra_status tra_build_block_mask(tra_plan p, const int32_t* radius_sq, uint8_t* mask,
                                int32_t* cnt, int32_t* cols, int32_t* order, void* workspace,
                                size_t workspace_bytes, void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_aligned4(radius_sq, "radius_sq", false));
  TRA_TRY(check_aligned4(cnt, "cnt", false));
  TRA_TRY(check_aligned4(cols, "cols", false));
  TRA_TRY(check_aligned4(order, "order", true));
  tra_plan_s bound;
  TRA_TRY(bind_workspace(p, TRA_CALL_BLOCK_MASK, order != nullptr, workspace, workspace_bytes, &bound));
  hipError_t e = tra::launch_block_mask(*p, radius_sq, mask, cnt, cols, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tra_build_block_mask launch");
  if (order) {
    e = tra::launch_row_order(bound, cnt, order, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "tra_build_block_mask order launch");
  }
  return ok();
}

tra_status tra_build_block_mask_noalloc(tra_plan p, const int32_t* radius_sq, uint8_t* mask,
                                        int32_t* cnt, int32_t* cols, int32_t* order, void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_aligned4(radius_sq, "radius_sq", false));
  TRA_TRY(check_aligned4(cnt, "cnt", false));
  TRA_TRY(check_aligned4(cols, "cols", false));
  TRA_TRY(check_aligned4(order, "order", true));
  const int64_t need = (int64_t)(p->NB + 1) * p->sort_chunks;
  if (order && need > tra::kNoAllocScratchInts)
    return fail(TRA_ERR_UNSUPPORTED,
                "tra_build_block_mask_noalloc: the row order needs " + std::to_string(need) +
                    " workspace ints, above the scratch array's " + std::to_string(tra::kNoAllocScratchInts) +
                    " ((NB + 1) * ceil(batch * heads * NB / 256) must stay within it)");
  hipError_t e = tra::launch_block_mask(*p, radius_sq, mask, cnt, cols, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "tra_build_block_mask_noalloc launch");
  if (order) {
    e = tra::launch_row_order_noalloc(*p, cnt, order, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "tra_build_block_mask_noalloc order launch");
  }
  return ok();
}

tra_status tra_sparse_attention(tra_plan p, const void* q, const void* k, const void* v,
                                const int32_t* cnt, const int32_t* cols, const int32_t* order,
                                void* o, float* lse, void* workspace, size_t workspace_bytes,
                                void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_tensor(q, "q"));
  TRA_TRY(check_tensor(k, "k"));
  TRA_TRY(check_tensor(v, "v"));
  TRA_TRY(check_tensor(o, "o"));
  TRA_TRY(check_aligned4(cnt, "cnt", false));
  TRA_TRY(check_aligned4(cols, "cols", false));
  TRA_TRY(check_aligned4(order, "order", true));
  TRA_TRY(check_aligned4(lse, "lse", true));
  tra::AttnArgs a{q, k, v, o, lse, nullptr, cnt, cols, order, true};
  return run_attention(p, TRA_CALL_SPARSE, a, workspace, workspace_bytes, stream, "tra_sparse_attention launch");
}

tra_status tra_token_attention(tra_plan p, const void* q, const void* k, const void* v,
                               const int32_t* radius_sq, const int32_t* cnt, const int32_t* cols,
                               const int32_t* order, void* o, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_tensor(q, "q"));
  TRA_TRY(check_tensor(k, "k"));
  TRA_TRY(check_tensor(v, "v"));
  TRA_TRY(check_tensor(o, "o"));
  TRA_TRY(check_aligned4(radius_sq, "radius_sq", false));
  TRA_TRY(check_aligned4(cnt, "cnt", false));
  TRA_TRY(check_aligned4(cols, "cols", false));
  TRA_TRY(check_aligned4(order, "order", true));
  TRA_TRY(check_aligned4(lse, "lse", true));
  if (p->cfg.dtype == TRA_BF16) {
    if (p->thr_max > 65535)
      return fail(TRA_ERR_UNSUPPORTED, "token attention on bf16 plans needs every threshold below 65536");
    if (p->cfg.block_layout == TRA_BLOCKS_PACKED && p->cfg.height * p->cfg.width < p->cfg.block)
      return fail(TRA_ERR_UNSUPPORTED, "token attention on bf16 plans needs height * width >= block");
  }
  tra::AttnArgs a{q, k, v, o, lse, nullptr, cnt, cols, order, true, radius_sq};
  return run_attention(p, TRA_CALL_TOKEN, a, workspace, workspace_bytes, stream, "tra_token_attention launch");
}

tra_status tra_dense_attention(tra_plan p, const void* q, const void* k, const void* v,
                               void* o, float* lse, void* workspace, size_t workspace_bytes,
                               void* stream) {
  TRA_TRY(check_plan(p));
  TRA_TRY(check_tensor(q, "q"));
  TRA_TRY(check_tensor(k, "k"));
  TRA_TRY(check_tensor(v, "v"));
  TRA_TRY(check_tensor(o, "o"));
  TRA_TRY(check_aligned4(lse, "lse", true));
  tra::AttnArgs a{q, k, v, o, lse, nullptr, nullptr, nullptr, nullptr, false};
  return run_attention(p, TRA_CALL_DENSE, a, workspace, workspace_bytes, stream, "tra_dense_attention launch");
}

}  // extern "C"

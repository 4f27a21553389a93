// C-ABI of the library (include/dcp.h): argument validation, workspace
// layout, path selection and kernel launches. Every check runs on the host
// before the first launch, so a rejected call touches neither the GPU nor the
// HIP runtime.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>

#include "dcp.h"
#include "dcp_internal.h"

namespace {

thread_local char g_err[512] = "";
thread_local void* g_ev_start = nullptr;
thread_local void* g_ev_stop = nullptr;

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return DCP_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

enum Path { kPathFast, kPathGeneric };

int check_shape(const dcp_shape* sh) {
  if (!sh) return fail(DCP_ERR_INVALID_ARGUMENT, "shape is NULL");
  if (sh->n_tokens < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "n_tokens must be >= 1 (got %lld)", (long long)sh->n_tokens);
  if (sh->c_s < 1 || sh->c_z < 1 || sh->n_heads < 1 || sh->head_dim < 1)
    return fail(DCP_ERR_INVALID_ARGUMENT, "c_s, c_z, n_heads and head_dim must be >= 1");
  if ((sh->act_dtype != DCP_F32 && sh->act_dtype != DCP_BF16) || (sh->out_dtype != DCP_F32 && sh->out_dtype != DCP_BF16))
    return fail(DCP_ERR_INVALID_ARGUMENT, "act_dtype and out_dtype must be DCP_F32 or DCP_BF16");
  if (!(sh->ln_eps >= 0.0f) || !isfinite(sh->ln_eps)) return fail(DCP_ERR_INVALID_ARGUMENT, "ln_eps must be finite and >= 0");
  if (sh->n_tokens > (int64_t)1 << 40) return fail(DCP_ERR_INVALID_ARGUMENT, "n_tokens too large");
  return DCP_OK;
}

int pick_path(const dcp_shape* sh, Path* p) {
  if (sh->act_dtype == DCP_BF16 && sh->c_z == dcp::kFastCz && sh->n_heads == dcp::kFastH &&
      sh->head_dim == dcp::kFastD && sh->c_s % 32 == 0 && sh->c_s <= dcp::kMaxCs &&
      sh->n_tokens <= dcp::kFastMaxTokens) {
    *p = kPathFast;
    return DCP_OK;
  }
  if (sh->c_z <= dcp::kGenMaxCz && sh->n_heads <= dcp::kGenMaxH && sh->head_dim <= dcp::kGenMaxD &&
      sh->n_heads * sh->head_dim <= dcp::kGenMaxHD && sh->c_s <= dcp::kMaxCs) {
    *p = kPathGeneric;
    return DCP_OK;
  }
  return fail(DCP_ERR_UNSUPPORTED,
              "unsupported shape (dtype %d, c_s %d, c_z %d, H %d, d %d): the fused path needs bf16, c_z=128, "
              "H=16, d=24, c_s%%32==0; the general path needs c_z<=256, H<=16, d<=64, H*d<=128, c_s<=4096",
              sh->act_dtype, sh->c_s, sh->c_z, sh->n_heads, sh->head_dim);
}

// Segments per key block for the fused kernel. A workgroup (kTileQ * 4 query
// rows) holds a whole CU (160 KB of LDS), so workgroups run in rounds of
// kSchedCUs, and a last round that fills only part of the chip leaves the rest
// idle for a whole workgroup's time. The cost of a choice, in units of one
// key streamed by one workgroup, is rounds x (keys per part + a fixed
// per-workgroup cost) plus the partial states it adds (H (d+2) fp32 per row and
// part, written then read by the merge: about 13 keys of z per row and part,
// spread over the chip). The smallest segment count within 2% of the cheapest
// is taken, so that more partials are only paid for a real gain. No part is
// longer than kMaxPartKeys keys: each part's fp32 accumulator is one sequential
// chain of per-tile matrix-core sums, and bounding its length bounds the
// rounding difference between two blockings of the same keys.
constexpr int64_t kSchedCUs = 256;     // CUs of an MI350X / MI355X (gfx950)
constexpr int64_t kMaxPartKeys = 4096;
constexpr int64_t kGroupCostKeys = 8;  // prologue (q, weights, ring fill) and epilogue, in keys
constexpr int64_t kPartCostKeys = 13;  // partial state per row and part, in keys of z per row

int fast_segments(int64_t n_tok, int64_t n_q, int32_t n_kb) {
  const int64_t groups = (n_q + 4 * dcp::kTileQ - 1) / (4 * dcp::kTileQ);
  const int64_t block = (n_tok + n_kb - 1) / n_kb;
  int64_t cap = (n_tok / n_kb) / 64;
  if (cap < 1) cap = 1;
  if (cap > 64) cap = 64;
  int64_t seg_min = (block + kMaxPartKeys - 1) / kMaxPartKeys;
  if (seg_min > cap) seg_min = cap;
  double cost[65];
  double best = 0.0;
  for (int64_t seg = seg_min; seg <= cap; ++seg) {
    const int64_t wgs = groups * n_kb * seg;
    const int64_t rounds = (wgs + kSchedCUs - 1) / kSchedCUs;
    const int64_t keys = (block + seg - 1) / seg;
    cost[seg] = (double)rounds * (double)(keys + kGroupCostKeys) +
                (double)n_q * (double)(n_kb * seg) * kPartCostKeys / (64.0 * kSchedCUs);
    if (seg == seg_min || cost[seg] < best) best = cost[seg];
  }
  for (int64_t seg = seg_min; seg <= cap; ++seg)
    if (cost[seg] <= 1.02 * best) return (int)seg;
  return (int)seg_min;
}

struct Layout {
  Path path;
  int n_seg, n_parts;
  int64_t nq_pad, n_pad;
  size_t off_q, off_k, off_v, off_tv, off_ws, off_g, off_m, off_l, off_acc, total;
};

void make_layout(const dcp_shape* sh, Path path, int64_t n_q, int32_t n_kb, Layout* L) {
  const int64_t hd = (int64_t)sh->n_heads * sh->head_dim;
  L->path = path;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = round_up(off + bytes, 256);
    return o;
  };
  if (path == kPathFast) {
    L->n_seg = fast_segments(sh->n_tokens, n_q, n_kb);
    L->n_parts = n_kb * L->n_seg;
    L->nq_pad = (n_q + 15) / 16 * 16;
    L->n_pad = (sh->n_tokens + 15) / 16 * 16;
    L->off_q = take((size_t)dcp::kFastH * L->nq_pad * dcp::kFastDp * 2);
    L->off_k = take((size_t)dcp::kFastH * L->n_pad * dcp::kFastDp * 2);
    L->off_v = take((size_t)dcp::kFastH * L->n_pad * dcp::kFastDp * 2);
    L->off_tv = take((size_t)(L->n_pad / 16) * 4);
    L->off_ws = take(dcp::fast_proj_split_bytes(sh->c_s));
  } else {
    L->n_seg = 1;
    L->n_parts = n_kb;
    L->nq_pad = n_q;
    L->n_pad = sh->n_tokens;
    L->off_q = take((size_t)n_q * hd * 4);
    L->off_k = take((size_t)sh->n_tokens * hd * 4);
    L->off_v = take((size_t)sh->n_tokens * hd * 4);
    L->off_tv = 0;
    L->off_ws = 0;
  }
  L->off_g = take((size_t)n_q * hd * 4);
  L->off_m = take((size_t)L->n_parts * sh->n_heads * n_q * 4);
  L->off_l = take((size_t)L->n_parts * sh->n_heads * n_q * 4);
  L->off_acc = take((size_t)L->n_parts * n_q * hd * 4);
  L->total = off;
}

int check_call(const dcp_shape* sh, int64_t n_q, int32_t n_kb, Path* path) {
  int rc = check_shape(sh);
  if (rc) return rc;
  if (n_q < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_q must be >= 0 (got %lld)", (long long)n_q);
  if (n_q > sh->n_tokens) return fail(DCP_ERR_INVALID_ARGUMENT, "n_q exceeds n_tokens");
  if (n_kb < 1 || n_kb > sh->n_tokens)
    return fail(DCP_ERR_INVALID_ARGUMENT, "n_key_blocks must be in [1, n_tokens] (got %d)", n_kb);
  return pick_path(sh, path);
}

}  // namespace

// Shared by the full call and the one-range partial: projections, the
// attention over keys [k_lo, k_lo + k_len) in n_key_blocks blocks, then the
// merge (into out, or into the partial state when `part` is set).
struct PartialOut {
  float *m, *l, *acc, *gate;
};
static int run_attention(const dcp_shape* shape, const dcp_weights* w, const void* s, const void* z_rows,
                         const uint8_t* key_mask, int64_t q_row0, int64_t n_q, int32_t n_key_blocks, int64_t k_lo,
                         int64_t k_len, void* out, const PartialOut* part, void* workspace, size_t workspace_bytes,
                         void* stream) {
  Path path;
  int rc = check_call(shape, n_q, n_key_blocks, &path);
  if (rc) return rc;
  if (q_row0 < 0 || q_row0 > shape->n_tokens - n_q)
    return fail(DCP_ERR_INVALID_ARGUMENT, "need 0 <= q_row0 and q_row0 + n_q <= n_tokens (q_row0 %lld, n_q %lld)",
                (long long)q_row0, (long long)n_q);
  if (!w) return fail(DCP_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->w_q || !w->w_k || !w->w_v || !w->w_g || !w->w_b)
    return fail(DCP_ERR_INVALID_ARGUMENT, "w_q, w_k, w_v, w_g and w_b are required");
  if (!s || !z_rows || (!out && !part)) return fail(DCP_ERR_INVALID_ARGUMENT, "s, z_rows and out are required");
  if (part && (!part->m || !part->l || !part->acc))
    return fail(DCP_ERR_INVALID_ARGUMENT, "m_out, l_out and acc_out are required");
  if (n_q == 0) return ok();
  if (!aligned(s, 16) || !aligned(z_rows, 16) || (out && !aligned(out, 16)))
    return fail(DCP_ERR_INVALID_ARGUMENT, "s, z_rows and out must be 16-byte aligned");
  if (part && (!aligned(part->m, 4) || !aligned(part->l, 4) || !aligned(part->acc, 4) ||
               (part->gate && !aligned(part->gate, 4))))
    return fail(DCP_ERR_INVALID_ARGUMENT, "m_out, l_out, acc_out and gate_out must be 4-byte aligned");
  if (path == kPathFast && (!aligned(w->w_q, 16) || !aligned(w->w_k, 16) || !aligned(w->w_v, 16) ||
                            !aligned(w->w_g, 16) || !aligned(w->w_b, 16) || !aligned(w->ln_gamma, 16)))
    return fail(DCP_ERR_INVALID_ARGUMENT, "w_q, w_k, w_v, w_g, w_b and ln_gamma must be 16-byte aligned");
  Layout L;
  make_layout(shape, path, n_q, n_key_blocks, &L);
  // a key range shorter than N: its own segment count, never more parts than
  // the layout holds, so the same workspace serves
  if (path == kPathFast && k_len < shape->n_tokens) {
    const int seg = fast_segments(k_len > 0 ? k_len : 1, n_q, n_key_blocks);
    if (seg < L.n_seg) L.n_seg = seg;
    L.n_parts = n_key_blocks * L.n_seg;
  }
  if (!workspace || !aligned(workspace, 256))
    return fail(DCP_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
  if (workspace_bytes < L.total)
    return fail(DCP_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, L.total);

  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t N = shape->n_tokens;
  const int hd = shape->n_heads * shape->head_dim;
  const bool act_bf16 = shape->act_dtype == DCP_BF16;
  hipError_t e;
  const int32_t log2_units = path == kPathFast ? 1 : 0;
  if (path == kPathFast) {
    dcp::FastProjArgs pa{};
    pa.s = static_cast<const uint16_t*>(s);
    pa.w_q = w->w_q;
    pa.w_k = w->w_k;
    pa.w_v = w->w_v;
    pa.w_g = w->w_g;
    pa.mask = key_mask;
    pa.n_tok = N;
    pa.q_row0 = q_row0;
    pa.n_q = n_q;
    pa.nq_pad = L.nq_pad;
    pa.n_pad = L.n_pad;
    pa.c_s = shape->c_s;
    pa.q = reinterpret_cast<uint16_t*>(ws + L.off_q);
    pa.k = reinterpret_cast<uint16_t*>(ws + L.off_k);
    pa.vt = reinterpret_cast<uint16_t*>(ws + L.off_v);
    pa.g = reinterpret_cast<float*>(ws + L.off_g);
    pa.tile_valid = reinterpret_cast<uint32_t*>(ws + L.off_tv);
    pa.w_split = ws + L.off_ws;
    if ((e = dcp::launch_fast_proj(pa, st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "projection launch failed: %s", hipGetErrorString(e));
    dcp::FastAttnArgs aa{};
    aa.z = static_cast<const uint16_t*>(z_rows);
    aa.mask = key_mask;
    aa.w_b = w->w_b;
    aa.gamma = w->ln_gamma;
    aa.q = pa.q;
    aa.k = pa.k;
    aa.vt = pa.vt;
    aa.tile_valid = pa.tile_valid;
    aa.n_tok = N;
    aa.n_q = n_q;
    aa.nq_pad = L.nq_pad;
    aa.n_pad = L.n_pad;
    aa.k_lo = k_lo;
    aa.k_len = k_len;
    aa.n_kb = n_key_blocks;
    aa.n_seg = L.n_seg;
    aa.eps = shape->ln_eps;
    aa.m_parts = reinterpret_cast<float*>(ws + L.off_m);
    aa.l_parts = reinterpret_cast<float*>(ws + L.off_l);
    aa.acc_parts = reinterpret_cast<float*>(ws + L.off_acc);
    if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
    if (k_len > 0 && (e = dcp::launch_fast_attn(aa, st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "attention launch failed: %s", hipGetErrorString(e));
    if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  } else {
    dcp::GenProjArgs pa{};
    pa.s = s;
    pa.s_bf16 = act_bf16;
    pa.w_q = w->w_q;
    pa.w_k = w->w_k;
    pa.w_v = w->w_v;
    pa.w_g = w->w_g;
    pa.n_tok = N;
    pa.q_row0 = q_row0;
    pa.n_q = n_q;
    pa.c_s = shape->c_s;
    pa.hd = hd;
    pa.q = reinterpret_cast<float*>(ws + L.off_q);
    pa.k = reinterpret_cast<float*>(ws + L.off_k);
    pa.v = reinterpret_cast<float*>(ws + L.off_v);
    pa.g = reinterpret_cast<float*>(ws + L.off_g);
    if ((e = dcp::launch_gen_proj(pa, st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "projection launch failed: %s", hipGetErrorString(e));
    dcp::GenAttnArgs aa{};
    aa.z = z_rows;
    aa.z_bf16 = act_bf16;
    aa.mask = key_mask;
    aa.w_b = w->w_b;
    aa.gamma = w->ln_gamma;
    aa.q = pa.q;
    aa.k = pa.k;
    aa.v = pa.v;
    aa.n_tok = N;
    aa.n_q = n_q;
    aa.c_z = shape->c_z;
    aa.n_heads = shape->n_heads;
    aa.head_dim = shape->head_dim;
    aa.k_lo = k_lo;
    aa.k_len = k_len;
    aa.n_kb = n_key_blocks;
    aa.eps = shape->ln_eps;
    aa.m_parts = reinterpret_cast<float*>(ws + L.off_m);
    aa.l_parts = reinterpret_cast<float*>(ws + L.off_l);
    aa.acc_parts = reinterpret_cast<float*>(ws + L.off_acc);
    if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
    if (k_len > 0 && (e = dcp::launch_gen_attn(aa, st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "attention launch failed: %s", hipGetErrorString(e));
    if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  }
  dcp::MergeArgs ma{};
  ma.n_parts = k_len > 0 ? L.n_parts : 0;  // an empty range merges to the empty state
  ma.n_heads = shape->n_heads;
  ma.head_dim = shape->head_dim;
  ma.n_rows = n_q;
  ma.m = reinterpret_cast<const float*>(ws + L.off_m);
  ma.l = reinterpret_cast<const float*>(ws + L.off_l);
  ma.acc = reinterpret_cast<const float*>(ws + L.off_acc);
  ma.log2_units = log2_units;
  if (part) {
    ma.m_out = part->m;
    ma.l_out = part->l;
    ma.acc_out = part->acc;
    ma.m_natural = 1;
    if (part->gate && (e = hipMemcpyAsync(part->gate, ws + L.off_g, (size_t)n_q * hd * sizeof(float),
                                          hipMemcpyDeviceToDevice, st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "gate copy failed: %s", hipGetErrorString(e));
  } else {
    ma.gate = reinterpret_cast<const float*>(ws + L.off_g);
    ma.out = out;
    ma.out_bf16 = shape->out_dtype == DCP_BF16;
  }
  if ((e = dcp::launch_merge(ma, st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  return ok();
}

// ---- scratch of the entry point that allocates nothing
// One array per GPU the library runs on, held until the process ends. In host
// code `scratch` names a host-side stand-in, never the device memory: host
// code uses only the address hipGetSymbolAddress returns for each device.
static __device__ __align__(256) unsigned char scratch[DCP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch address on the current device, looked up once per device.
int scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(DCP_ERR_UNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(DCP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DCP_OK;
}

}  // namespace

extern "C" {

const char* dcp_last_error(void) { return g_err; }

const char* dcp_version(void) { return "dcp-mi355x 0.1 (gfx950)"; }

int dcp_set_timing_events(void* start_event, void* stop_event) {
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(DCP_ERR_INVALID_ARGUMENT, "timing events must both be set or both be NULL");
  g_ev_start = start_event;
  g_ev_stop = stop_event;
  return ok();
}

int dcp_workspace_size(const dcp_shape* shape, int64_t n_q, int32_t n_key_blocks, size_t* bytes) {
  if (!bytes) return fail(DCP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  Path path;
  const int rc = check_call(shape, n_q, n_key_blocks, &path);
  if (rc) return rc;
  if (n_q == 0) {
    *bytes = 0;
    return ok();
  }
  Layout L;
  make_layout(shape, path, n_q, n_key_blocks, &L);
  *bytes = L.total;
  return ok();
}

size_t dcp_workspace_bytes(const dcp_shape* shape, int64_t n_q, int32_t n_key_blocks) {
  size_t bytes = 0;
  if (!shape) {
    fail(DCP_ERR_INVALID_ARGUMENT, "shape is NULL");
    return 0;
  }
  if (n_q == 0) {
    // a valid no-op needs no workspace; an invalid shape still reports why
    Path path;
    if (check_call(shape, n_q, n_key_blocks, &path) != DCP_OK) return 0;
    ok();
    return 0;
  }
  return dcp_workspace_size(shape, n_q, n_key_blocks, &bytes) == DCP_OK ? bytes : 0;
}

int dcp_pair_bias_attention(const dcp_shape* shape, const dcp_weights* w, const void* s, const void* z_rows,
                            const uint8_t* key_mask, int64_t q_row0, int64_t n_q, int32_t n_key_blocks, void* out,
                            void* workspace, size_t workspace_bytes, void* stream) {
  return run_attention(shape, w, s, z_rows, key_mask, q_row0, n_q, n_key_blocks, 0, shape ? shape->n_tokens : 0, out,
                       nullptr, workspace, workspace_bytes, stream);
}

int dcp_pair_bias_attention_noalloc(const dcp_shape* shape, const dcp_weights* w, const void* s, const void* z_rows,
                                    const uint8_t* key_mask, int64_t q_row0, int64_t n_q, int32_t n_key_blocks,
                                    void* out, void* stream) {
  // every size check first: an oversized call touches neither the GPU nor the runtime
  size_t need = 0;
  int rc = dcp_workspace_size(shape, n_q, n_key_blocks, &need);
  if (rc) return rc;
  if (need > (size_t)DCP_NOALLOC_SCRATCH_BYTES)
    return fail(DCP_ERR_WORKSPACE,
                "the call needs %zu bytes of scratch, beyond the %zu-byte maximum of "
                "dcp_pair_bias_attention_noalloc; split the query rows into smaller stripes or use "
                "dcp_pair_bias_attention with a workspace",
                need, (size_t)DCP_NOALLOC_SCRATCH_BYTES);
  if (n_q == 0) return run_attention(shape, w, s, z_rows, key_mask, q_row0, n_q, n_key_blocks, 0,
                                     shape->n_tokens, out, nullptr, nullptr, 0, stream);
  if (stream) {
    int sdev = -1, cdev = -1;
    hipError_t e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
    if (e == hipSuccess) e = hipGetDevice(&cdev);
    if (e != hipSuccess) return fail(DCP_ERR_HIP, "stream device query failed: %s", hipGetErrorString(e));
    if (sdev != cdev)
      return fail(DCP_ERR_INVALID_ARGUMENT, "the stream belongs to device %d, the current device is %d", sdev, cdev);
  }
  void* ptr = nullptr;
  if ((rc = scratch_on_current_device(&ptr)) != DCP_OK) return rc;
  return run_attention(shape, w, s, z_rows, key_mask, q_row0, n_q, n_key_blocks, 0, shape->n_tokens, out, nullptr,
                       ptr, (size_t)DCP_NOALLOC_SCRATCH_BYTES, stream);
}

int dcp_pair_bias_attention_partial(const dcp_shape* shape, const dcp_weights* w, const void* s, const void* z_rows,
                                    const uint8_t* key_mask, int64_t q_row0, int64_t n_q, int64_t k0, int64_t k1,
                                    float* m_out, float* l_out, float* acc_out, float* gate_out, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  if (!shape) return fail(DCP_ERR_INVALID_ARGUMENT, "shape is NULL");
  if (k0 < 0 || k1 < k0 || k1 > shape->n_tokens)
    return fail(DCP_ERR_INVALID_ARGUMENT, "need 0 <= k0 <= k1 <= n_tokens (k0 %lld, k1 %lld)", (long long)k0,
                (long long)k1);
  const PartialOut part{m_out, l_out, acc_out, gate_out};
  return run_attention(shape, w, s, z_rows, key_mask, q_row0, n_q, 1, k0, k1 - k0, nullptr, &part, workspace,
                       workspace_bytes, stream);
}

int dcp_bias_project(const dcp_shape* shape, const dcp_weights* w, const void* z_tile, int64_t n_rows, int64_t n_cols,
                     int64_t row_stride_elems, float* bias_out, void* stream) {
  if (!shape) return fail(DCP_ERR_INVALID_ARGUMENT, "shape is NULL");
  if (shape->c_z < 1 || shape->n_heads < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "c_z and n_heads must be >= 1");
  if (shape->act_dtype != DCP_F32 && shape->act_dtype != DCP_BF16)
    return fail(DCP_ERR_INVALID_ARGUMENT, "act_dtype must be DCP_F32 or DCP_BF16");
  if (!(shape->ln_eps >= 0.0f) || !isfinite(shape->ln_eps)) return fail(DCP_ERR_INVALID_ARGUMENT, "ln_eps must be finite and >= 0");
  if (n_rows < 0 || n_cols < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_rows and n_cols must be >= 0");
  if (!w || !w->w_b) return fail(DCP_ERR_INVALID_ARGUMENT, "w_b is required");
  if (!z_tile || !bias_out) return fail(DCP_ERR_INVALID_ARGUMENT, "z_tile and bias_out are required");
  if (row_stride_elems < n_cols * (int64_t)shape->c_z)
    return fail(DCP_ERR_INVALID_ARGUMENT, "row_stride_elems must be >= n_cols * c_z");
  const bool fast = shape->act_dtype == DCP_BF16 && shape->c_z == dcp::kFastCz && shape->n_heads == dcp::kFastH;
  if (!fast && (shape->c_z > dcp::kGenMaxCz || shape->n_heads > dcp::kGenMaxH))
    return fail(DCP_ERR_UNSUPPORTED, "unsupported bias shape (c_z %d, H %d)", shape->c_z, shape->n_heads);
  if (n_rows == 0 || n_cols == 0) return ok();
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (fast) {
    if (!aligned(z_tile, 16) || !aligned(bias_out, 16) || row_stride_elems % 8 != 0)
      return fail(DCP_ERR_INVALID_ARGUMENT, "z_tile and bias_out must be 16-byte aligned, row_stride_elems a multiple of 8");
    if (!aligned(w->w_b, 16) || !aligned(w->ln_gamma, 16) || !aligned(w->ln_beta, 16))
      return fail(DCP_ERR_INVALID_ARGUMENT, "w_b, ln_gamma and ln_beta must be 16-byte aligned");
    dcp::FastBiasArgs a{};
    a.z = static_cast<const uint16_t*>(z_tile);
    a.w_b = w->w_b;
    a.b_b = w->b_b;
    a.gamma = w->ln_gamma;
    a.beta = w->ln_beta;
    a.n_rows = n_rows;
    a.n_cols = n_cols;
    a.row_stride = row_stride_elems;
    a.cols_per_wave = 64;
    a.eps = shape->ln_eps;
    a.out = bias_out;
    e = dcp::launch_fast_bias(a, st);
  } else {
    if (!aligned(bias_out, 4)) return fail(DCP_ERR_INVALID_ARGUMENT, "bias_out must be 4-byte aligned");
    dcp::GenBiasArgs a{};
    a.z = z_tile;
    a.z_bf16 = shape->act_dtype == DCP_BF16;
    a.w_b = w->w_b;
    a.b_b = w->b_b;
    a.gamma = w->ln_gamma;
    a.beta = w->ln_beta;
    a.n_rows = n_rows;
    a.n_cols = n_cols;
    a.row_stride = row_stride_elems;
    a.c_z = shape->c_z;
    a.n_heads = shape->n_heads;
    a.eps = shape->ln_eps;
    a.out = bias_out;
    e = dcp::launch_gen_bias(a, st);
  }
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "bias launch failed: %s", hipGetErrorString(e));
  return ok();
}

int dcp_block_merge(int32_t n_parts, int64_t n_rows, int32_t n_heads, int32_t head_dim, const float* m_parts,
                    const float* l_parts, const float* acc_parts, float* m_out, float* l_out, float* acc_out,
                    const float* gate, void* out, int32_t out_dtype, void* stream) {
  if (n_parts < 1 || n_heads < 1 || head_dim < 1 || n_rows < 0)
    return fail(DCP_ERR_INVALID_ARGUMENT, "need n_parts, n_heads, head_dim >= 1 and n_rows >= 0");
  if ((int64_t)n_heads * head_dim > 4096) return fail(DCP_ERR_UNSUPPORTED, "H*d must be <= 4096");
  if (out_dtype != DCP_F32 && out_dtype != DCP_BF16)
    return fail(DCP_ERR_INVALID_ARGUMENT, "out_dtype must be DCP_F32 or DCP_BF16");
  if (!m_parts || !l_parts || !acc_parts) return fail(DCP_ERR_INVALID_ARGUMENT, "m_parts, l_parts and acc_parts are required");
  if (n_rows == 0) return ok();
  dcp::MergeArgs a{};
  a.n_parts = n_parts;
  a.n_heads = n_heads;
  a.head_dim = head_dim;
  a.n_rows = n_rows;
  a.m = m_parts;
  a.l = l_parts;
  a.acc = acc_parts;
  a.gate = gate;
  a.m_out = m_out;
  a.l_out = l_out;
  a.acc_out = acc_out;
  a.out = out;
  a.out_bf16 = out_dtype == DCP_BF16;
  a.log2_units = 0;
  const hipError_t e = dcp::launch_merge(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

// ----------------------------------------------------------------------------- sparse atom attention
namespace {

struct SparseLayout {
  size_t off_q, off_g, off_k, off_v, total;
};

int check_sparse(const dcp_sparse_shape* sh, int64_t n_q) {
  if (!sh) return fail(DCP_ERR_INVALID_ARGUMENT, "shape is NULL");
  if (sh->n_atoms < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "n_atoms must be >= 1 (got %lld)", (long long)sh->n_atoms);
  if (sh->c_atom < 1 || sh->c_ap < 1 || sh->n_heads < 1 || sh->head_dim < 1 || sh->k < 1)
    return fail(DCP_ERR_INVALID_ARGUMENT, "c_atom, c_ap, n_heads, head_dim and k must be >= 1");
  if ((sh->act_dtype != DCP_F32 && sh->act_dtype != DCP_BF16) || (sh->out_dtype != DCP_F32 && sh->out_dtype != DCP_BF16))
    return fail(DCP_ERR_INVALID_ARGUMENT, "act_dtype and out_dtype must be DCP_F32 or DCP_BF16");
  if (sh->p_gathered != 0 && sh->p_gathered != 1) return fail(DCP_ERR_INVALID_ARGUMENT, "p_gathered must be 0 or 1");
  if (!(sh->ln_eps >= 0.0f) || !isfinite(sh->ln_eps)) return fail(DCP_ERR_INVALID_ARGUMENT, "ln_eps must be finite and >= 0");
  if (n_q < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_q must be >= 0 (got %lld)", (long long)n_q);
  if (n_q > sh->n_atoms) return fail(DCP_ERR_INVALID_ARGUMENT, "n_q exceeds n_atoms");
  if (sh->n_heads != dcp::kSparseH || sh->head_dim != dcp::kSparseD || sh->c_ap != dcp::kSparseCap ||
      sh->k > dcp::kSparseMaxK || sh->n_atoms > dcp::kSparseMaxAtoms || sh->c_atom > dcp::kMaxCs ||
      (sh->act_dtype == DCP_BF16 && sh->c_atom % 32 != 0))
    return fail(DCP_ERR_UNSUPPORTED,
                "unsupported sparse shape (H %d, d %d, c_ap %d, k %d, L %lld, c_atom %d, dtype %d): needs H=4, d=32, "
                "c_ap=16, k<=256, L<=4000000, c_atom<=4096 (a multiple of 32 for bf16)",
                sh->n_heads, sh->head_dim, sh->c_ap, sh->k, (long long)sh->n_atoms, sh->c_atom, sh->act_dtype);
  return DCP_OK;
}

void sparse_layout(const dcp_sparse_shape* sh, int64_t n_q, SparseLayout* L) {
  const size_t hd = (size_t)dcp::kSparseH * dcp::kSparseD;
  const size_t eb = sh->act_dtype == DCP_BF16 ? 2 : 4;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = round_up(off + bytes, 256);
    return o;
  };
  L->off_q = take((size_t)n_q * hd * 4);
  L->off_g = take((size_t)n_q * hd * 4);
  L->off_k = take((size_t)sh->n_atoms * hd * eb);
  L->off_v = take((size_t)sh->n_atoms * hd * eb);
  L->total = off;
}

}  // namespace

extern "C" {

int dcp_sparse_workspace_size(const dcp_sparse_shape* shape, int64_t n_q, size_t* bytes) {
  if (!bytes) return fail(DCP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  const int rc = check_sparse(shape, n_q);
  if (rc) return rc;
  if (n_q == 0) {
    *bytes = 0;
    return ok();
  }
  SparseLayout L;
  sparse_layout(shape, n_q, &L);
  *bytes = L.total;
  return ok();
}

int dcp_sparse_pair_bias_attention(const dcp_sparse_shape* shape, const dcp_weights* w, const void* a, const void* p,
                                   const int32_t* nbr, int64_t q_row0, int64_t n_q, int32_t n_key_blocks, void* out,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_sparse(shape, n_q);
  if (rc) return rc;
  if (q_row0 < 0 || q_row0 > shape->n_atoms - n_q)
    return fail(DCP_ERR_INVALID_ARGUMENT, "need 0 <= q_row0 and q_row0 + n_q <= n_atoms (q_row0 %lld, n_q %lld)",
                (long long)q_row0, (long long)n_q);
  if (n_key_blocks < 1 || n_key_blocks > shape->n_atoms)
    return fail(DCP_ERR_INVALID_ARGUMENT, "n_key_blocks must be in [1, n_atoms] (got %d)", n_key_blocks);
  if (!w) return fail(DCP_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!w->w_q || !w->w_k || !w->w_v || !w->w_g || !w->w_b)
    return fail(DCP_ERR_INVALID_ARGUMENT, "w_q, w_k, w_v, w_g and w_b are required");
  if (!a || !p || !nbr || !out) return fail(DCP_ERR_INVALID_ARGUMENT, "a, p, nbr and out are required");
  if (n_q == 0) return ok();
  if (!aligned(a, 16) || !aligned(p, 16) || !aligned(out, 16) || !aligned(nbr, 4))
    return fail(DCP_ERR_INVALID_ARGUMENT, "a, p and out must be 16-byte aligned, nbr 4-byte aligned");
  const bool bf16 = shape->act_dtype == DCP_BF16;
  if (bf16 && (!aligned(w->w_q, 16) || !aligned(w->w_k, 16) || !aligned(w->w_v, 16) || !aligned(w->w_g, 16)))
    return fail(DCP_ERR_INVALID_ARGUMENT, "w_q, w_k, w_v and w_g must be 16-byte aligned");
  SparseLayout L;
  sparse_layout(shape, n_q, &L);
  if (!workspace || !aligned(workspace, 256))
    return fail(DCP_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
  if (workspace_bytes < L.total)
    return fail(DCP_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, L.total);

  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (bf16) {
    dcp::SparseProjArgs pa{};
    pa.a = static_cast<const uint16_t*>(a);
    pa.w_q = w->w_q;
    pa.w_k = w->w_k;
    pa.w_v = w->w_v;
    pa.w_g = w->w_g;
    pa.n_atoms = shape->n_atoms;
    pa.q_row0 = q_row0;
    pa.n_q = n_q;
    pa.c_atom = shape->c_atom;
    pa.q = reinterpret_cast<float*>(ws + L.off_q);
    pa.g = reinterpret_cast<float*>(ws + L.off_g);
    pa.k = reinterpret_cast<uint16_t*>(ws + L.off_k);
    pa.v = reinterpret_cast<uint16_t*>(ws + L.off_v);
    e = dcp::launch_sparse_proj(pa, st);
  } else {
    dcp::GenProjArgs pa{};
    pa.s = a;
    pa.s_bf16 = 0;
    pa.w_q = w->w_q;
    pa.w_k = w->w_k;
    pa.w_v = w->w_v;
    pa.w_g = w->w_g;
    pa.n_tok = shape->n_atoms;
    pa.q_row0 = q_row0;
    pa.n_q = n_q;
    pa.c_s = shape->c_atom;
    pa.hd = dcp::kSparseH * dcp::kSparseD;
    pa.q = reinterpret_cast<float*>(ws + L.off_q);
    pa.k = reinterpret_cast<float*>(ws + L.off_k);
    pa.v = reinterpret_cast<float*>(ws + L.off_v);
    pa.g = reinterpret_cast<float*>(ws + L.off_g);
    e = dcp::launch_gen_proj(pa, st);
  }
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "projection launch failed: %s", hipGetErrorString(e));

  dcp::SparseAttnArgs aa{};
  aa.p = p;
  aa.nbr = nbr;
  aa.w_b = w->w_b;
  aa.gamma = w->ln_gamma;
  aa.q = reinterpret_cast<const float*>(ws + L.off_q);
  aa.g = reinterpret_cast<const float*>(ws + L.off_g);
  aa.k = ws + L.off_k;
  aa.v = ws + L.off_v;
  aa.n_atoms = shape->n_atoms;
  aa.n_q = n_q;
  aa.p_row_elems = (shape->p_gathered ? (int64_t)shape->k : shape->n_atoms) * shape->c_ap;
  aa.k_slots = shape->k;
  aa.n_kb = n_key_blocks;
  aa.p_gathered = shape->p_gathered;
  aa.out_bf16 = shape->out_dtype == DCP_BF16;
  aa.eps = shape->ln_eps;
  aa.out = out;
  if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  if ((e = dcp::launch_sparse_attn(aa, bf16, st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "sparse attention launch failed: %s", hipGetErrorString(e));
  if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  return ok();
}

// ----------------------------------------------------------------------------- k nearest neighbours
int dcp_knn_workspace_size(int64_t n_c, size_t* bytes) {
  if (!bytes) return fail(DCP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_c < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_c must be >= 0");
  *bytes = dcp::knn_workspace_bytes(n_c, nullptr);
  return ok();
}

int dcp_knn_topk(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, int64_t c_index0, int64_t q_self0,
                 const int32_t* group_q, const int32_t* group_c, int32_t group_mode, int32_t k, int32_t* idx_out,
                 float* d2_out, void* workspace, size_t workspace_bytes, void* stream) {
  if (n_q < 0 || n_c < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_q and n_c must be >= 0");
  if (k < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "k must be >= 1 (got %d)", k);
  if (k > dcp::kKnnMaxK) return fail(DCP_ERR_UNSUPPORTED, "k must be <= %d (got %d)", dcp::kKnnMaxK, k);
  if (c_index0 < 0 || c_index0 + n_c > (int64_t)INT32_MAX)
    return fail(DCP_ERR_INVALID_ARGUMENT, "candidate indices c_index0 .. c_index0 + n_c must fit in int32");
  if (group_mode < 0 || group_mode > 2) return fail(DCP_ERR_INVALID_ARGUMENT, "group_mode must be 0, 1 or 2");
  if (group_mode != 0 && (!group_q || !group_c))
    return fail(DCP_ERR_INVALID_ARGUMENT, "group_q and group_c are required when group_mode != 0");
  if (n_q == 0) return ok();
  if (!x_q || (!x_c && n_c > 0) || !idx_out)
    return fail(DCP_ERR_INVALID_ARGUMENT, "x_q, x_c (when n_c > 0) and idx_out are required");
  if (!aligned(x_q, 4) || !aligned(x_c, 4) || !aligned(idx_out, 4) || (d2_out && !aligned(d2_out, 4)))
    return fail(DCP_ERR_INVALID_ARGUMENT, "x_q, x_c, idx_out and d2_out must be 4-byte aligned");
  size_t box_offset = 0;
  const size_t need = dcp::knn_workspace_bytes(n_c, &box_offset);
  if (n_c > 0 && (!workspace || !aligned(workspace, 256)))
    return fail(DCP_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
  if (n_c > 0 && workspace_bytes < need)
    return fail(DCP_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
  dcp::KnnArgs a{};
  a.x_q = x_q;
  a.x_c = x_c;
  a.group_q = group_q;
  a.group_c = group_c;
  a.n_q = n_q;
  a.n_c = n_c;
  a.c_index0 = c_index0;
  a.q_self0 = q_self0 >= 0 && q_self0 < n_c ? q_self0 : -1;
  a.k = k;
  a.group_mode = group_mode;
  a.idx_out = idx_out;
  a.d2_out = d2_out;
  a.cand = workspace;
  a.box = static_cast<char*>(workspace) + box_offset;
  hipError_t e;
  if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), static_cast<hipStream_t>(stream))) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  if ((e = dcp::launch_knn(a, static_cast<hipStream_t>(stream))) != hipSuccess)
    return fail(DCP_ERR_HIP, "knn launch failed: %s", hipGetErrorString(e));
  if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), static_cast<hipStream_t>(stream))) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  return ok();
}

int dcp_topk_merge(int64_t n_rows, int32_t k, const int32_t* idx_a, const float* d2_a, const int32_t* idx_b,
                   const float* d2_b, int32_t* idx_out, float* d2_out, void* stream) {
  if (n_rows < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_rows must be >= 0");
  if (k < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "k must be >= 1 (got %d)", k);
  if (k > dcp::kKnnMaxK) return fail(DCP_ERR_UNSUPPORTED, "k must be <= %d (got %d)", dcp::kKnnMaxK, k);
  if (!idx_a || !d2_a || !idx_b || !d2_b || !idx_out || !d2_out)
    return fail(DCP_ERR_INVALID_ARGUMENT, "all six lists are required");
  if (n_rows == 0) return ok();
  dcp::TopkMergeArgs a{};
  a.n_rows = n_rows;
  a.k = k;
  a.idx_a = idx_a;
  a.idx_b = idx_b;
  a.d2_a = d2_a;
  a.d2_b = d2_b;
  a.idx_out = idx_out;
  a.d2_out = d2_out;
  const hipError_t e = dcp::launch_topk_merge(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "top-k merge launch failed: %s", hipGetErrorString(e));
  return ok();
}

// ----------------------------------------------------------------------------- pair transition
static int check_transition(int32_t c_z, int32_t hidden, int32_t act_dtype, bool* fast) {
  if (c_z < 1 || hidden < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "c_z and hidden must be >= 1");
  if (act_dtype != DCP_F32 && act_dtype != DCP_BF16)
    return fail(DCP_ERR_INVALID_ARGUMENT, "act_dtype must be DCP_F32 or DCP_BF16");
  if (act_dtype == DCP_BF16) {
    if (c_z != dcp::kTransCz || hidden != dcp::kTransHidden)
      return fail(DCP_ERR_UNSUPPORTED, "bf16 transition needs c_z = %d and hidden = %d (got %d, %d)", dcp::kTransCz,
                  dcp::kTransHidden, c_z, hidden);
    *fast = true;
    return DCP_OK;
  }
  if (c_z > dcp::kGenMaxCz || hidden > dcp::kTransGenMaxHidden)
    return fail(DCP_ERR_UNSUPPORTED, "fp32 transition needs c_z <= %d and hidden <= %d", dcp::kGenMaxCz,
                dcp::kTransGenMaxHidden);
  *fast = false;
  return DCP_OK;
}

int dcp_transition_workspace_size(int32_t c_z, int32_t hidden, int32_t act_dtype, size_t* bytes) {
  if (!bytes) return fail(DCP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  bool fast;
  const int rc = check_transition(c_z, hidden, act_dtype, &fast);
  if (rc) return rc;
  *bytes = fast ? round_up(dcp::trans_prep_bytes(), 256) : 0;
  return ok();
}

int dcp_pair_transition(int64_t n_pairs, int32_t c_z, int32_t hidden, int32_t act_dtype, float ln_eps,
                        const float* w1, const float* w2, const float* w3, const float* ln_gamma,
                        const float* ln_beta, const void* z_in, void* z_out, void* workspace, size_t workspace_bytes,
                        void* stream) {
  bool fast;
  int rc = check_transition(c_z, hidden, act_dtype, &fast);
  if (rc) return rc;
  if (n_pairs < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_pairs must be >= 0");
  if (!(ln_eps >= 0.0f) || !isfinite(ln_eps)) return fail(DCP_ERR_INVALID_ARGUMENT, "ln_eps must be finite and >= 0");
  if (!w1 || !w2 || !w3) return fail(DCP_ERR_INVALID_ARGUMENT, "w1, w2 and w3 are required");
  if (!z_in || !z_out) return fail(DCP_ERR_INVALID_ARGUMENT, "z_in and z_out are required");
  if (n_pairs == 0) return ok();
  if (!aligned(z_in, 16) || !aligned(z_out, 16))
    return fail(DCP_ERR_INVALID_ARGUMENT, "z_in and z_out must be 16-byte aligned");
  const size_t zbytes = (size_t)n_pairs * c_z * (act_dtype == DCP_BF16 ? 2 : 4);
  const char *zi = static_cast<const char*>(z_in), *zo = static_cast<const char*>(z_out);
  if (zi != zo && zi < zo + zbytes && zo < zi + zbytes)
    return fail(DCP_ERR_INVALID_ARGUMENT, "z_out must equal z_in or not overlap it");
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (fast) {
    const size_t need = round_up(dcp::trans_prep_bytes(), 256);
    if (!workspace || !aligned(workspace, 256))
      return fail(DCP_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
    if (workspace_bytes < need)
      return fail(DCP_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
    dcp::TransArgs a{};
    a.n_pairs = n_pairs;
    a.w1 = w1;
    a.w2 = w2;
    a.w3 = w3;
    a.gamma = ln_gamma;
    a.beta = ln_beta;
    a.z_in = z_in;
    a.z_out = z_out;
    a.w_prep = workspace;
    a.gb_prep = reinterpret_cast<float*>(static_cast<char*>(workspace) + (dcp::trans_prep_bytes() - 2 * dcp::kTransCz * sizeof(float)));
    a.eps = ln_eps;
    if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
    e = dcp::launch_transition(a, st);
  } else {
    dcp::TransGenArgs a{};
    a.n_pairs = n_pairs;
    a.c_z = c_z;
    a.hidden = hidden;
    a.w1 = w1;
    a.w2 = w2;
    a.w3 = w3;
    a.gamma = ln_gamma;
    a.beta = ln_beta;
    a.z_in = static_cast<const float*>(z_in);
    a.z_out = static_cast<float*>(z_out);
    a.eps = ln_eps;
    if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
      return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
    e = dcp::launch_transition_gen(a, st);
  }
  if (e != hipSuccess) return fail(DCP_ERR_HIP, "transition launch failed: %s", hipGetErrorString(e));
  if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  return ok();
}

// ----------------------------------------------------------------------------- atom -> token mean
static size_t scatter_ws(int64_t n_tokens, int32_t c) {
  return round_up((size_t)n_tokens * c * 8, 256) + round_up((size_t)n_tokens * 4, 256) +
         round_up(dcp::kScatterFlags * sizeof(int32_t), 256) + round_up((size_t)n_tokens * 16, 256);
}

static int check_scatter(int64_t n_atoms, int64_t n_tokens, int32_t c, int32_t in_dtype, int32_t out_dtype) {
  if (n_atoms < 0 || n_tokens < 0) return fail(DCP_ERR_INVALID_ARGUMENT, "n_atoms and n_tokens must be >= 0");
  if (c < 1) return fail(DCP_ERR_INVALID_ARGUMENT, "c must be >= 1");
  if (c > dcp::kScatterMaxC) return fail(DCP_ERR_UNSUPPORTED, "c must be <= %d (got %d)", dcp::kScatterMaxC, c);
  if ((in_dtype != DCP_F32 && in_dtype != DCP_BF16) || (out_dtype != DCP_F32 && out_dtype != DCP_BF16))
    return fail(DCP_ERR_INVALID_ARGUMENT, "dtypes must be DCP_F32 or DCP_BF16");
  return DCP_OK;
}

int dcp_scatter_mean_workspace_size(int64_t n_tokens, int32_t c, size_t* bytes) {
  if (!bytes) return fail(DCP_ERR_INVALID_ARGUMENT, "bytes is NULL");
  const int rc = check_scatter(0, n_tokens, c, DCP_F32, DCP_F32);
  if (rc) return rc;
  *bytes = n_tokens == 0 ? 0 : scatter_ws(n_tokens, c);
  return ok();
}

int dcp_scatter_mean(int64_t n_atoms, int64_t n_tokens, int32_t c, int32_t in_dtype, int32_t out_dtype, const void* a,
                     const int32_t* tok_idx, void* out, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_scatter(n_atoms, n_tokens, c, in_dtype, out_dtype);
  if (rc) return rc;
  if (n_tokens == 0) return ok();
  if (!out || (n_atoms > 0 && (!a || !tok_idx)))
    return fail(DCP_ERR_INVALID_ARGUMENT, "out (and a, tok_idx when n_atoms > 0) are required");
  const size_t ea = in_dtype == DCP_BF16 ? 2 : 4, eo = out_dtype == DCP_BF16 ? 2 : 4;
  if ((a && !aligned(a, ea)) || (tok_idx && !aligned(tok_idx, 4)) || !aligned(out, eo))
    return fail(DCP_ERR_INVALID_ARGUMENT, "a, tok_idx and out must be aligned to their element size");
  const size_t need = scatter_ws(n_tokens, c);
  if (!workspace || !aligned(workspace, 256))
    return fail(DCP_ERR_WORKSPACE, "workspace must be a 256-byte aligned device pointer");
  if (workspace_bytes < need)
    return fail(DCP_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
  dcp::ScatterArgs s{};
  s.n_atoms = n_atoms;
  s.n_tokens = n_tokens;
  s.c = c;
  s.a_bf16 = in_dtype == DCP_BF16;
  s.out_bf16 = out_dtype == DCP_BF16;
  s.a = a;
  s.tok_idx = tok_idx;
  s.acc = static_cast<int64_t*>(workspace);
  s.cnt = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + round_up((size_t)n_tokens * c * 8, 256));
  s.flags = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(s.cnt) + round_up((size_t)n_tokens * 4, 256));
  s.plan = reinterpret_cast<int64_t*>(reinterpret_cast<char*>(s.flags) + round_up(dcp::kScatterFlags * sizeof(int32_t), 256));
  s.out = out;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (g_ev_start && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_start), st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  if ((e = dcp::launch_scatter_mean(s, st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "scatter-mean launch failed: %s", hipGetErrorString(e));
  if (g_ev_stop && (e = hipEventRecord(static_cast<hipEvent_t>(g_ev_stop), st)) != hipSuccess)
    return fail(DCP_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

// C-ABI entry points: argument validation, workspace layout and kernel
// launches on the caller's stream. No device allocation and no host sync on
// the hot path; rp_validate_layout is the one test utility that does both.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "rp.h"
#include "rp_internal.h"

namespace {

thread_local char g_err[512];

rp_status fail(rp_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

rp_status hip_fail(hipError_t e, const char* what) {
  return fail(RP_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Shape {
  int S, G, Hq, Hkv, D, nrep, max_pp, max_rp, num_pages;
  bool fp8;
};

rp_status check_kv(const rp_paged_kv* kv) {
  if (kv == nullptr) return fail(RP_ERR_INVALID_ARG, "kv is NULL");
  if (kv->k_pages == nullptr || kv->v_pages == nullptr) return fail(RP_ERR_INVALID_ARG, "k_pages/v_pages is NULL");
  if (!aligned(kv->k_pages, 16) || !aligned(kv->v_pages, 16))
    return fail(RP_ERR_INVALID_ARG, "k_pages/v_pages must be 16-byte aligned");
  if (kv->num_pages < 1) return fail(RP_ERR_INVALID_ARG, "num_pages must be >= 1 (got %d)", kv->num_pages);
  if (kv->num_kv_heads < 1) return fail(RP_ERR_INVALID_ARG, "num_kv_heads must be >= 1");
  if (kv->page_size != rp::kPage) return fail(RP_ERR_UNSUPPORTED, "page_size %d unsupported (16 only)", kv->page_size);
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(RP_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", kv->head_dim);
  const int dtype = rp::enum_bits(kv->kv_dtype);
  if (dtype == RP_KV_BF16) {
    if (kv->k_scale != nullptr || kv->v_scale != nullptr)
      return fail(RP_ERR_INVALID_ARG, "k_scale/v_scale must be NULL for bf16 KV");
  } else if (dtype == RP_KV_FP8_E4M3) {
    if (kv->k_scale == nullptr || kv->v_scale == nullptr)
      return fail(RP_ERR_INVALID_ARG, "k_scale/v_scale required for fp8 KV");
    if (!aligned(kv->k_scale, 4) || !aligned(kv->v_scale, 4))
      return fail(RP_ERR_INVALID_ARG, "k_scale/v_scale must be 4-byte aligned");
  } else {
    return fail(RP_ERR_UNSUPPORTED, "kv_dtype %d unsupported", dtype);
  }
  return RP_OK;
}

rp_status check_shape(const rp_paged_kv* kv, const rp_group_layout* l, Shape* sh) {
  rp_status st = check_kv(kv);
  if (st != RP_OK) return st;
  if (l == nullptr) return fail(RP_ERR_INVALID_ARG, "layout is NULL");
  if (l->num_seqs < 0) return fail(RP_ERR_INVALID_ARG, "num_seqs must be >= 0");
  if (l->num_q_heads < 1) return fail(RP_ERR_INVALID_ARG, "num_q_heads must be >= 1");
  if (l->num_q_heads % kv->num_kv_heads != 0)
    return fail(RP_ERR_INVALID_ARG, "num_q_heads %d not a multiple of num_kv_heads %d", l->num_q_heads,
                kv->num_kv_heads);
  const int nrep = l->num_q_heads / kv->num_kv_heads;
  if (nrep != 1 && nrep != 2 && nrep != 4 && nrep != 8)
    return fail(RP_ERR_UNSUPPORTED, "q/kv head ratio %d unsupported (1, 2, 4, 8)", nrep);
  if (l->max_prefix_pages < 0 || l->max_resp_pages < 0)
    return fail(RP_ERR_INVALID_ARG, "table widths must be >= 0");
  if (l->num_seqs > 0) {
    if (l->num_groups < 1) return fail(RP_ERR_INVALID_ARG, "num_groups must be >= 1");
    if (l->seq_to_group == nullptr || l->prefix_lens == nullptr || l->resp_lens == nullptr)
      return fail(RP_ERR_INVALID_ARG, "seq_to_group/prefix_lens/resp_lens is NULL");
    if (l->max_prefix_pages > 0 && l->prefix_block_table == nullptr)
      return fail(RP_ERR_INVALID_ARG, "prefix_block_table is NULL");
    if (l->max_resp_pages > 0 && l->resp_block_table == nullptr)
      return fail(RP_ERR_INVALID_ARG, "resp_block_table is NULL");
  }
  // Every index the kernels form stays below 2^31 elements per int32 table.
  const long long rows = (long long)l->num_seqs * l->num_q_heads;
  if (l->num_seqs > 0 && l->num_groups > rp::kPlanMaxGroups)
    return fail(RP_ERR_UNSUPPORTED, "num_groups %d above the planner's limit %d", l->num_groups, rp::kPlanMaxGroups);
  if ((long long)l->num_seqs * l->max_resp_pages >= (1ll << 31) ||
      (long long)l->num_groups * l->max_prefix_pages >= (1ll << 31) || rows >= (1ll << 31))
    return fail(RP_ERR_UNSUPPORTED, "layout too large for int32 indexing");
  sh->S = l->num_seqs;
  sh->G = l->num_groups;
  sh->Hq = l->num_q_heads;
  sh->Hkv = kv->num_kv_heads;
  sh->D = kv->head_dim;
  sh->nrep = nrep;
  sh->max_pp = l->max_prefix_pages;
  sh->max_rp = l->max_resp_pages;
  sh->num_pages = kv->num_pages;
  sh->fp8 = rp::enum_bits(kv->kv_dtype) == RP_KV_FP8_E4M3;
  return RP_OK;
}

// Workspace layout, 256-byte aligned sections.
struct WsLayout {
  size_t hdr, grp_off, members, pitems, ritems, seq_parts, part_o, part_lse, total;
  long long max_pitems, max_ritems, max_parts;
  int max_pc, max_rc;
};

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

bool ws_layout(const Shape& sh, WsLayout* w) {
  w->max_pc = rp::cdiv(sh.max_pp, rp::kPrefixChunkPages);
  const bool small = (long long)sh.S * sh.max_rp * sh.Hkv <= rp::kSmallBatchPageHeads;
  w->max_rc = rp::cdiv(sh.max_rp, small ? rp::kRespChunkPagesSmall : rp::kRespChunkPagesMin);
  const long long groups_used = sh.G < sh.S ? sh.G : sh.S;
  w->max_pitems = groups_used * w->max_pc;
  w->max_ritems = (long long)sh.S * w->max_rc;
  w->max_parts = (long long)sh.S * sh.Hq * (w->max_pc + w->max_rc);
  if (w->max_parts >= (1ll << 31) || w->max_ritems * sh.Hkv >= (1ll << 31) ||
      w->max_pitems * sh.Hkv >= (1ll << 31))
    return false;
  size_t o = 0;
  w->hdr = o;       o = align_up(o + sizeof(int) * rp::kHdrSlots);
  w->grp_off = o;   o = align_up(o + sizeof(int) * ((size_t)sh.G + 1));
  w->members = o;   o = align_up(o + sizeof(int) * (size_t)sh.S);
  w->pitems = o;    o = align_up(o + sizeof(int2) * (size_t)w->max_pitems);
  w->ritems = o;    o = align_up(o + sizeof(int4) * (size_t)w->max_ritems);
  w->seq_parts = o; o = align_up(o + sizeof(int) * (size_t)sh.S);
  w->part_o = o;    o = align_up(o + sizeof(float) * (size_t)w->max_parts * sh.D);
  w->part_lse = o;  o = align_up(o + sizeof(float) * (size_t)w->max_parts);
  w->total = o;
  return true;
}

// Compute units of the current device, queried once per device (racing first
// calls store the same value; relaxed atomics keep that race defined).
rp_status device_cus(int* cus) {
  static std::atomic<int> cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(RP_ERR_UNSUPPORTED, "device %d out of range", dev);
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    cache[dev].store(n, std::memory_order_relaxed);
  }
  *cus = n;
  return RP_OK;
}

// Scratch of rp_group_decode_attn_noalloc: the work plan and partial results
// live in this device array instead of a caller workspace. Each GPU holds its
// own copy for the life of the process; its name is only a host-side handle,
// so host code uses the device address looked up once per device below.
__device__ __align__(256) static unsigned char scratch[RP_NOALLOC_SCRATCH_BYTES];

rp_status scratch_address(void** out) {
  static std::atomic<void*> addr[64];
  static std::mutex lookup;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(RP_ERR_UNSUPPORTED, "device %d out of range", dev);
  void* p = addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(lookup);
    p = addr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // with device `dev` current
      if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
      if (p == nullptr || !aligned(p, 256)) return fail(RP_ERR_HIP, "scratch has no usable device address");
      addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return RP_OK;
}

rp::PlanView plan_view(void* ws, const WsLayout& w) {
  char* b = static_cast<char*>(ws);
  rp::PlanView v;
  v.hdr = reinterpret_cast<int*>(b + w.hdr);
  v.grp_off = reinterpret_cast<int*>(b + w.grp_off);
  v.grp_members = reinterpret_cast<int*>(b + w.members);
  v.prefix_items = reinterpret_cast<int2*>(b + w.pitems);
  v.resp_items = reinterpret_cast<int4*>(b + w.ritems);
  v.seq_parts = reinterpret_cast<int*>(b + w.seq_parts);
  v.part_o = reinterpret_cast<float*>(b + w.part_o);
  v.part_lse = reinterpret_cast<float*>(b + w.part_lse);
  v.max_prefix_chunks = w.max_pc;
  v.max_resp_chunks = w.max_rc;
  v.parts_per_row = w.max_pc + w.max_rc;
  v.max_parts = (int)w.max_parts;
  v.max_prefix_items = (int)w.max_pitems;
  v.max_resp_items = (int)w.max_ritems;
  return v;
}

rp_status prepare(const rp_paged_kv* kv, const rp_group_layout* l, void* ws, size_t ws_bytes, Shape* sh,
                  WsLayout* w) {
  rp_status st = check_shape(kv, l, sh);
  if (st != RP_OK) return st;
  if (!ws_layout(*sh, w)) return fail(RP_ERR_UNSUPPORTED, "layout too large for the work plan");
  if (sh->S == 0) return RP_OK;
  if (ws == nullptr) return fail(RP_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(RP_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < w->total)
    return fail(RP_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, w->total);
  return RP_OK;
}

rp::AttnArgs attn_args(const rp_paged_kv* kv, const rp_group_layout* l, const void* q, float scale,
                       const rp::PlanView& v) {
  rp::AttnArgs a;
  a.k_pages = kv->k_pages;
  a.v_pages = kv->v_pages;
  a.k_scale = kv->k_scale;
  a.v_scale = kv->v_scale;
  a.num_pages = kv->num_pages;
  a.num_kv_heads = kv->num_kv_heads;
  a.num_seqs = l->num_seqs;
  a.num_groups = l->num_groups;
  a.num_q_heads = l->num_q_heads;
  a.seq_to_group = l->seq_to_group;
  a.prefix_lens = l->prefix_lens;
  a.prefix_block_table = l->prefix_block_table;
  a.max_prefix_pages = l->max_prefix_pages;
  a.resp_lens = l->resp_lens;
  a.resp_block_table = l->resp_block_table;
  a.max_resp_pages = l->max_resp_pages;
  a.q = q;
  a.qk_scale = scale * rp::kLog2e;
  a.view = v;
  return a;
}

// The planner's arguments for a prepared batch (queries the device's compute
// units, which set the piece length).
rp_status plan_args(const Shape& sh, const rp_group_layout* l, void* ws, const WsLayout& w, int len_add,
                    rp::PlanArgs* a) {
  int cus = 0;
  rp_status st = device_cus(&cus);
  if (st != RP_OK) return st;
  a->num_seqs = sh.S;
  a->num_groups = sh.G;
  a->num_q_heads = sh.Hq;
  a->num_kv_heads = sh.Hkv;
  a->num_cus = cus;
  a->seq_to_group = l->seq_to_group;
  a->prefix_lens = l->prefix_lens;
  a->resp_lens = l->resp_lens;
  a->len_add = len_add;
  a->max_prefix_pages = sh.max_pp;
  a->max_resp_pages = sh.max_rp;
  a->view = plan_view(ws, w);
  return RP_OK;
}

// Checks and launch arguments of the decode step's q/k prep.
rp_status qk_prep_args(const rp_paged_kv* kv, const rp_group_layout* l, const Shape& sh, const void* q_in,
                       const void* k_in, const void* v_in, const void* q_norm_w, const void* k_norm_w,
                       double rms_eps, double rope_theta, void* q_out, void* k_out, rp::QkPrepArgs* a) {
  if (!(rms_eps >= 0.0) || !std::isfinite(rms_eps)) return fail(RP_ERR_INVALID_ARG, "rms_eps must be finite and >= 0");
  if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
    return fail(RP_ERR_INVALID_ARG, "rope_theta must be finite and > 0");
  if (sh.S == 0) return RP_OK;
  const void* in[] = {q_in, k_in, v_in, q_norm_w, k_norm_w, q_out};
  for (const void* p : in)
    if (p == nullptr || !aligned(p, 16))
      return fail(RP_ERR_INVALID_ARG, "q_in/k_in/v_in/q_norm_w/k_norm_w/q_out must be non-NULL and 16-byte aligned");
  if (k_out != nullptr && !aligned(k_out, 16)) return fail(RP_ERR_INVALID_ARG, "k_out must be 16-byte aligned");
  if (sh.max_rp < 1) return fail(RP_ERR_INVALID_ARG, "max_resp_pages must be >= 1 to append");
  a->k_pages = kv->k_pages;
  a->v_pages = kv->v_pages;
  a->k_scale = kv->k_scale;
  a->v_scale = kv->v_scale;
  a->num_pages = kv->num_pages;
  a->num_kv_heads = sh.Hkv;
  a->num_q_heads = sh.Hq;
  a->num_seqs = sh.S;
  a->num_groups = sh.G;
  a->seq_to_group = l->seq_to_group;
  a->prefix_lens = l->prefix_lens;
  a->resp_lens = l->resp_lens;
  a->resp_block_table = l->resp_block_table;
  a->max_resp_pages = sh.max_rp;
  a->q_in = static_cast<const uint16_t*>(q_in);
  a->k_in = static_cast<const uint16_t*>(k_in);
  a->v_in = static_cast<const uint16_t*>(v_in);
  a->q_norm_w = static_cast<const uint16_t*>(q_norm_w);
  a->k_norm_w = static_cast<const uint16_t*>(k_norm_w);
  a->rms_eps = rms_eps;
  // Rotary frequencies on the host in fp64 (libm pow), passed with the arguments.
  for (int i = 0; i < rp::kMaxHeadDim / 2; ++i)
    a->inv_freq[i] = i < sh.D / 2 ? std::pow(rope_theta, (-2.0 * i) / sh.D) : 0.0;
  a->q_out = static_cast<uint16_t*>(q_out);
  a->k_out = static_cast<uint16_t*>(k_out);
  a->blocks_per_seq = 0;
  return RP_OK;
}

}  // namespace

extern "C" {

const char* rp_status_string(rp_status status) {
  switch (rp::enum_bits(status)) {
    case RP_OK: return "RP_OK: success";
    case RP_ERR_INVALID_ARG: return "RP_ERR_INVALID_ARG: invalid argument";
    case RP_ERR_UNSUPPORTED: return "RP_ERR_UNSUPPORTED: unsupported configuration";
    case RP_ERR_WORKSPACE: return "RP_ERR_WORKSPACE: workspace missing or too small";
    case RP_ERR_HIP: return "RP_ERR_HIP: HIP runtime error";
    case RP_ERR_LAYOUT: return "RP_ERR_LAYOUT: layout entry out of range";
  }
  return "unknown rp_status";
}

const char* rp_last_error(void) { return g_err; }

rp_status rp_group_decode_attn_workspace_size(const rp_paged_kv* kv, const rp_group_layout* layout,
                                              size_t* bytes) {
  g_err[0] = 0;
  if (bytes == nullptr) return fail(RP_ERR_INVALID_ARG, "bytes is NULL");
  Shape sh;
  rp_status st = check_shape(kv, layout, &sh);
  if (st != RP_OK) return st;
  WsLayout w;
  if (!ws_layout(sh, &w)) return fail(RP_ERR_UNSUPPORTED, "layout too large for the work plan");
  *bytes = sh.S == 0 ? 0 : w.total;
  return RP_OK;
}

rp_status rp_plan(const rp_paged_kv* kv, const rp_group_layout* l, void* ws, size_t ws_bytes,
                  hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  WsLayout w;
  rp_status st = prepare(kv, l, ws, ws_bytes, &sh, &w);
  if (st != RP_OK || sh.S == 0) return st;
  rp::PlanArgs a;
  st = plan_args(sh, l, ws, w, 0, &a);
  if (st != RP_OK) return st;
  hipError_t e = rp::launch_plan(a, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "plan kernel launch");
}

rp_status rp_attn_parts(const rp_paged_kv* kv, const rp_group_layout* l, const void* q, float softmax_scale,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  WsLayout w;
  rp_status st = prepare(kv, l, ws, ws_bytes, &sh, &w);
  if (st != RP_OK || sh.S == 0) return st;
  if (q == nullptr || !aligned(q, 16)) return fail(RP_ERR_INVALID_ARG, "q must be non-NULL and 16-byte aligned");
  const rp::AttnArgs a = attn_args(kv, l, q, softmax_scale, plan_view(ws, w));
  hipError_t e = rp::launch_attn_parts(a, sh.D, sh.nrep, sh.fp8, w.max_pitems, w.max_ritems, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "attention parts kernel launch");
}

rp_status rp_combine_parts(const rp_paged_kv* kv, const rp_group_layout* l, void* out, float* lse, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  WsLayout w;
  rp_status st = prepare(kv, l, ws, ws_bytes, &sh, &w);
  if (st != RP_OK || sh.S == 0) return st;
  if (out == nullptr || !aligned(out, 16)) return fail(RP_ERR_INVALID_ARG, "out must be non-NULL and 16-byte aligned");
  if (lse != nullptr && !aligned(lse, 4)) return fail(RP_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  const rp::PlanView v = plan_view(ws, w);
  rp::CombineArgs c{};
  c.o_parts = v.part_o;
  c.lse_parts = v.part_lse;
  c.row_offs = nullptr;
  c.num_rows = sh.S * sh.Hq;
  c.out = out;
  c.lse = lse;
  c.seq_parts = v.seq_parts;
  c.num_q_heads = sh.Hq;
  c.parts_per_row = v.parts_per_row;
  hipError_t e = rp::launch_combine(c, sh.D, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "combine kernel launch");
}

rp_status rp_group_decode_attn(const rp_paged_kv* kv, const rp_group_layout* l, const void* q,
                               float softmax_scale, void* out, float* lse, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  WsLayout w;
  rp_status st = prepare(kv, l, ws, ws_bytes, &sh, &w);
  if (st != RP_OK || sh.S == 0) return st;
  if (q == nullptr || !aligned(q, 16)) return fail(RP_ERR_INVALID_ARG, "q must be non-NULL and 16-byte aligned");
  if (out == nullptr || !aligned(out, 16)) return fail(RP_ERR_INVALID_ARG, "out must be non-NULL and 16-byte aligned");
  if (lse != nullptr && !aligned(lse, 4)) return fail(RP_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  st = rp_plan(kv, l, ws, ws_bytes, stream);
  if (st != RP_OK) return st;
  st = rp_attn_parts(kv, l, q, softmax_scale, ws, ws_bytes, stream);
  if (st != RP_OK) return st;
  return rp_combine_parts(kv, l, out, lse, ws, ws_bytes, stream);
}

rp_status rp_group_decode_attn_noalloc(const rp_paged_kv* kv, const rp_group_layout* l, const void* q,
                                       float softmax_scale, void* out, float* lse, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  rp_status st = check_shape(kv, l, &sh);
  if (st != RP_OK) return st;
  WsLayout w;
  if (!ws_layout(sh, &w)) return fail(RP_ERR_UNSUPPORTED, "layout too large for the work plan");
  if (sh.S == 0) return RP_OK;
  if (w.total > (size_t)RP_NOALLOC_SCRATCH_BYTES)
    return fail(RP_ERR_WORKSPACE,
                "this layout needs %zu bytes of scratch; the library's static scratch holds %zu "
                "(use rp_group_decode_attn with a workspace)",
                w.total, (size_t)RP_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != RP_OK) return st;
  // The same three launches as rp_group_decode_attn. The plan overwrites every
  // entry the attention and combine kernels read, so nothing needs clearing.
  return rp_group_decode_attn(kv, l, q, softmax_scale, out, lse, ws, RP_NOALLOC_SCRATCH_BYTES, stream);
}

rp_status rp_lse_combine(const float* o_parts, const float* lse_parts, const int32_t* row_part_offsets,
                         int32_t num_rows, int32_t head_dim, void* out, float* lse_out, hipStream_t stream) {
  g_err[0] = 0;
  if (num_rows < 0) return fail(RP_ERR_INVALID_ARG, "num_rows must be >= 0");
  if (head_dim != 64 && head_dim != 128) return fail(RP_ERR_UNSUPPORTED, "head_dim %d unsupported", head_dim);
  if (num_rows == 0) return RP_OK;
  if (row_part_offsets == nullptr || out == nullptr)
    return fail(RP_ERR_INVALID_ARG, "row_part_offsets/out is NULL");
  if (!aligned(out, 8)) return fail(RP_ERR_INVALID_ARG, "out must be 8-byte aligned");
  if (lse_out != nullptr && !aligned(lse_out, 4)) return fail(RP_ERR_INVALID_ARG, "lse_out must be 4-byte aligned");
  if ((o_parts != nullptr && !aligned(o_parts, 16)) || (lse_parts != nullptr && !aligned(lse_parts, 4)))
    return fail(RP_ERR_INVALID_ARG, "o_parts must be 16-byte and lse_parts 4-byte aligned");
  rp::CombineArgs c{};
  c.o_parts = o_parts;
  c.lse_parts = lse_parts;
  c.row_offs = row_part_offsets;
  c.num_rows = num_rows;
  c.out = out;
  c.lse = lse_out;
  hipError_t e = rp::launch_combine(c, head_dim, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "combine kernel launch");
}

rp_status rp_kv_append(const rp_paged_kv* kv, const rp_group_layout* l, const void* k_new, const void* v_new,
                       hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  rp_status st = check_shape(kv, l, &sh);
  if (st != RP_OK) return st;
  if (sh.S == 0) return RP_OK;
  if (k_new == nullptr || v_new == nullptr || !aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(RP_ERR_INVALID_ARG, "k_new/v_new must be non-NULL and 16-byte aligned");
  if (sh.max_rp < 1) return fail(RP_ERR_INVALID_ARG, "max_resp_pages must be >= 1 to append");
  rp::AppendArgs a;
  a.k_pages = kv->k_pages;
  a.v_pages = kv->v_pages;
  a.k_scale = kv->k_scale;
  a.v_scale = kv->v_scale;
  a.num_pages = kv->num_pages;
  a.num_kv_heads = kv->num_kv_heads;
  a.num_seqs = sh.S;
  a.resp_lens = l->resp_lens;
  a.resp_block_table = l->resp_block_table;
  a.max_resp_pages = sh.max_rp;
  a.k_new = k_new;
  a.v_new = v_new;
  hipError_t e = rp::launch_append(a, sh.D, sh.fp8, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "append kernel launch");
}

rp_status rp_decode_qk_prep(const rp_paged_kv* kv, const rp_group_layout* l, const void* q_in, const void* k_in,
                            const void* v_in, const void* q_norm_w, const void* k_norm_w, double rms_eps,
                            double rope_theta, void* q_out, void* k_out, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  rp_status st = check_shape(kv, l, &sh);
  if (st != RP_OK) return st;
  rp::QkPrepArgs a;
  st = qk_prep_args(kv, l, sh, q_in, k_in, v_in, q_norm_w, k_norm_w, rms_eps, rope_theta, q_out, k_out, &a);
  if (st != RP_OK || sh.S == 0) return st;
  hipError_t e = rp::launch_qk_prep(a, sh.D, sh.fp8, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "decode q/k prep kernel launch");
}

rp_status rp_decode_qk_prep_plan(const rp_paged_kv* kv, const rp_group_layout* l, const void* q_in,
                                 const void* k_in, const void* v_in, const void* q_norm_w, const void* k_norm_w,
                                 double rms_eps, double rope_theta, void* q_out, void* k_out, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  WsLayout w;
  rp_status st = prepare(kv, l, ws, ws_bytes, &sh, &w);
  if (st != RP_OK) return st;
  rp::QkPrepArgs a;
  st = qk_prep_args(kv, l, sh, q_in, k_in, v_in, q_norm_w, k_norm_w, rms_eps, rope_theta, q_out, k_out, &a);
  if (st != RP_OK || sh.S == 0) return st;
  rp::PlanArgs p;
  st = plan_args(sh, l, ws, w, 1, &p);
  if (st != RP_OK) return st;
  hipError_t e;
  if (sh.S <= rp::kSmallPlanMaxSeqs && sh.G <= rp::kPlanMaxGroups) {
    e = rp::launch_qk_prep_plan(a, p, sh.D, sh.fp8, stream);
    return e == hipSuccess ? RP_OK : hip_fail(e, "decode q/k prep + plan kernel launch");
  }
  e = rp::launch_qk_prep(a, sh.D, sh.fp8, stream);
  if (e != hipSuccess) return hip_fail(e, "decode q/k prep kernel launch");
  e = rp::launch_plan(p, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "plan kernel launch");
}

rp_status rp_grpo_advantage(const float* rewards, int32_t num_groups, int32_t group_size, double eps_std,
                            int32_t ddof, float* advantages, float* group_mean, float* group_std,
                            hipStream_t stream) {
  g_err[0] = 0;
  if (num_groups < 0 || group_size < 1)
    return fail(RP_ERR_INVALID_ARG, "num_groups must be >= 0 and group_size >= 1");
  if (ddof != 0 && ddof != 1) return fail(RP_ERR_INVALID_ARG, "ddof must be 0 or 1");
  if (!(eps_std >= 0.0) || !std::isfinite(eps_std)) return fail(RP_ERR_INVALID_ARG, "eps_std must be finite and >= 0");
  if ((long long)num_groups * group_size >= (1ll << 40)) return fail(RP_ERR_UNSUPPORTED, "too many rewards");
  if (num_groups == 0) return RP_OK;
  if (rewards == nullptr || advantages == nullptr || !aligned(rewards, 4) || !aligned(advantages, 4))
    return fail(RP_ERR_INVALID_ARG, "rewards/advantages must be non-NULL fp32 arrays");
  if ((group_mean != nullptr && !aligned(group_mean, 4)) || (group_std != nullptr && !aligned(group_std, 4)))
    return fail(RP_ERR_INVALID_ARG, "group_mean/group_std must be fp32 arrays");
  rp::GrpoArgs a;
  a.rewards = rewards;
  a.num_groups = num_groups;
  a.group_size = group_size;
  a.ddof = ddof;
  a.eps_std = eps_std;
  a.advantages = advantages;
  a.mean = group_mean;
  a.stdev = group_std;
  a.vector_ok = aligned(rewards, 16) && aligned(advantages, 16);
  hipError_t e = rp::launch_grpo(a, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "GRPO advantage kernel launch");
}

// Shared checks of the prefill calls; fills a (pointers of the projections
// and outputs are checked by the callers).
static rp_status prefill_args(const rp_paged_kv* kv, const rp_prefill_layout* l, rp::PrefillArgs* a, int* n_rep) {
  rp_status st = check_kv(kv);
  if (st != RP_OK) return st;
  if (l == nullptr) return fail(RP_ERR_INVALID_ARG, "layout is NULL");
  if (l->num_groups < 0 || l->num_tokens < 0) return fail(RP_ERR_INVALID_ARG, "num_groups/num_tokens must be >= 0");
  if (l->num_q_heads < 1 || l->num_q_heads % kv->num_kv_heads != 0)
    return fail(RP_ERR_INVALID_ARG, "num_q_heads %d not a positive multiple of num_kv_heads %d", l->num_q_heads,
                kv->num_kv_heads);
  const int r = l->num_q_heads / kv->num_kv_heads;
  if (r != 1 && r != 2 && r != 4 && r != 8)
    return fail(RP_ERR_UNSUPPORTED, "q/kv head ratio %d unsupported (1, 2, 4, 8)", r);
  if (l->num_groups > 0) {
    if (l->prompt_offs == nullptr) return fail(RP_ERR_INVALID_ARG, "prompt_offs is NULL");
    if (l->max_prefix_pages < 1 || l->prefix_block_table == nullptr)
      return fail(RP_ERR_INVALID_ARG, "prefix_block_table must be non-NULL with max_prefix_pages >= 1");
  }
  // One prompt's K/V rows are addressed with 32-bit byte offsets.
  if ((long long)l->num_groups * l->max_prefix_pages * kv->num_kv_heads >= (1ll << 31) ||
      (long long)l->num_tokens * l->num_q_heads * kv->head_dim >= (1ll << 40) ||
      (long long)l->max_prefix_pages * rp::kPage * kv->num_kv_heads * kv->head_dim * 2 >= (1ll << 32))
    return fail(RP_ERR_UNSUPPORTED, "prefill too large");
  a->k_pages = kv->k_pages;
  a->v_pages = kv->v_pages;
  a->k_scale = kv->k_scale;
  a->v_scale = kv->v_scale;
  a->num_pages = kv->num_pages;
  a->num_kv_heads = kv->num_kv_heads;
  a->num_groups = l->num_groups;
  a->num_q_heads = l->num_q_heads;
  a->num_tokens = l->num_tokens;
  a->prompt_offs = l->prompt_offs;
  a->prefix_block_table = l->prefix_block_table;
  a->max_prefix_pages = l->max_prefix_pages;
  *n_rep = r;
  return RP_OK;
}

rp_status rp_prefill_kv_write(const rp_paged_kv* kv, const rp_prefill_layout* l, const void* k, const void* v,
                              hipStream_t stream) {
  g_err[0] = 0;
  rp::PrefillArgs a{};
  int n_rep = 0;
  rp_status st = prefill_args(kv, l, &a, &n_rep);
  if (st != RP_OK) return st;
  if (l->num_groups == 0 || l->num_tokens == 0) return RP_OK;
  if (k == nullptr || v == nullptr || !aligned(k, 16) || !aligned(v, 16))
    return fail(RP_ERR_INVALID_ARG, "k/v must be non-NULL and 16-byte aligned");
  a.k = k;
  a.v = v;
  hipError_t e = rp::launch_prefill_kv_write(a, kv->head_dim, rp::enum_bits(kv->kv_dtype) == RP_KV_FP8_E4M3, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "prefill KV write kernel launch");
}

// Causal attention within each prompt; with `pages`, also the prompts' K/V
// page writes: in the same launch for bf16 pools, by the page-write kernel
// first for fp8 pools (their per-page scales need a whole page).
static rp_status prefill_impl(const rp_paged_kv* kv, const rp_prefill_layout* l, const void* q, const void* k,
                              const void* v, float softmax_scale, void* out, float* lse, bool pages,
                              hipStream_t stream) {
  g_err[0] = 0;
  rp::PrefillArgs a{};
  int n_rep = 0;
  rp_status st = prefill_args(kv, l, &a, &n_rep);
  if (st != RP_OK) return st;
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    return fail(RP_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  if (l->num_groups == 0 || l->num_tokens == 0) return RP_OK;
  if (q == nullptr || k == nullptr || v == nullptr || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16))
    return fail(RP_ERR_INVALID_ARG, "q/k/v must be non-NULL and 16-byte aligned");
  if (out == nullptr || !aligned(out, 16)) return fail(RP_ERR_INVALID_ARG, "out must be non-NULL and 16-byte aligned");
  if (lse != nullptr && !aligned(lse, 4)) return fail(RP_ERR_INVALID_ARG, "lse must be 4-byte aligned");
  a.q = q;
  a.k = k;
  a.v = v;
  a.qk_scale = softmax_scale * rp::kLog2e;
  a.out = out;
  a.lse = lse;
  const bool fp8 = rp::enum_bits(kv->kv_dtype) == RP_KV_FP8_E4M3;
  if (pages && fp8) {
    hipError_t e = rp::launch_prefill_kv_write(a, kv->head_dim, true, stream);
    if (e != hipSuccess) return hip_fail(e, "prefill KV write kernel launch");
  }
  a.write_pages = pages && !fp8 ? 1 : 0;
  hipError_t e = rp::launch_prefill_attn(a, kv->head_dim, n_rep, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "prefill attention kernel launch");
}

rp_status rp_prefill_attn(const rp_paged_kv* kv, const rp_prefill_layout* l, const void* q, const void* k,
                          const void* v, float softmax_scale, void* out, float* lse, hipStream_t stream) {
  return prefill_impl(kv, l, q, k, v, softmax_scale, out, lse, false, stream);
}

rp_status rp_prefill(const rp_paged_kv* kv, const rp_prefill_layout* l, const void* q, const void* k, const void* v,
                     float softmax_scale, void* out, float* lse, hipStream_t stream) {
  return prefill_impl(kv, l, q, k, v, softmax_scale, out, lse, true, stream);
}

rp_status rp_plan_layout(const rp_paged_kv* kv, const rp_group_layout* l, rp_plan_info* info) {
  g_err[0] = 0;
  if (info == nullptr) return fail(RP_ERR_INVALID_ARG, "info is NULL");
  Shape sh;
  rp_status st = check_shape(kv, l, &sh);
  if (st != RP_OK) return st;
  WsLayout w;
  if (!ws_layout(sh, &w)) return fail(RP_ERR_UNSUPPORTED, "layout too large for the work plan");
  info->hdr = w.hdr;
  info->grp_off = w.grp_off;
  info->grp_members = w.members;
  info->prefix_items = w.pitems;
  info->resp_items = w.ritems;
  info->seq_parts = w.seq_parts;
  info->part_o = w.part_o;
  info->part_lse = w.part_lse;
  info->max_prefix_items = (int32_t)w.max_pitems;
  info->max_resp_items = (int32_t)w.max_ritems;
  info->parts_per_row = w.max_pc + w.max_rc;
  info->max_parts = (int32_t)w.max_parts;
  return RP_OK;
}

rp_status rp_validate_layout(const rp_paged_kv* kv, const rp_group_layout* l, hipStream_t stream) {
  g_err[0] = 0;
  Shape sh;
  rp_status st = check_shape(kv, l, &sh);
  if (st != RP_OK) return st;
  if (sh.S == 0) return RP_OK;
  int* dres = nullptr;
  hipError_t e = hipMalloc(&dres, 4 * sizeof(int));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc");
  int hres[4] = {0, 0, 0, 0};
  e = hipMemcpyAsync(dres, hres, sizeof(hres), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) {
    rp::ValidateArgs a;
    a.num_pages = sh.num_pages;
    a.num_seqs = sh.S;
    a.num_groups = sh.G;
    a.seq_to_group = l->seq_to_group;
    a.prefix_lens = l->prefix_lens;
    a.prefix_block_table = l->prefix_block_table;
    a.max_prefix_pages = sh.max_pp;
    a.resp_lens = l->resp_lens;
    a.resp_block_table = l->resp_block_table;
    a.max_resp_pages = sh.max_rp;
    a.result = dres;
    e = rp::launch_validate(a, stream);
  }
  if (e == hipSuccess) e = hipMemcpyAsync(hres, dres, sizeof(hres), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  hipError_t ef = hipFree(dres);
  if (e != hipSuccess) return hip_fail(e, "validate_layout");
  if (ef != hipSuccess) return hip_fail(ef, "hipFree");
  if (hres[0] != 0) {
    static const char* kinds[] = {"?", "seq_to_group", "prefix_lens", "resp_lens", "prefix_block_table",
                                  "resp_block_table"};
    const int k = (hres[1] >= 1 && hres[1] <= 5) ? hres[1] : 0;
    return fail(RP_ERR_LAYOUT, "%d bad entries; e.g. %s at index %d has value %d", hres[0], kinds[k], hres[2],
                hres[3]);
  }
  return RP_OK;
}

rp_status rp_selftest_mfma(int32_t shape, const void* a, const void* b, float* c, hipStream_t stream) {
  g_err[0] = 0;
  if (shape < RP_SELFTEST_MFMA_16X16X32 || shape > RP_SELFTEST_MFMA_16X16X32_LDS_TR)
    return fail(RP_ERR_UNSUPPORTED, "self-test shape %d unknown", shape);
  if (a == nullptr || b == nullptr || c == nullptr) return fail(RP_ERR_INVALID_ARG, "a/b/c is NULL");
  if (!aligned(a, 2) || !aligned(b, 2) || !aligned(c, 4))
    return fail(RP_ERR_INVALID_ARG, "a and b must be 2-byte and c 4-byte aligned");
  hipError_t e = rp::launch_selftest_mfma(shape, a, b, c, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "self-test kernel launch");
}

rp_status rp_stream_read(const void* src, uint64_t bytes, uint32_t* sink, int32_t nontemporal, hipStream_t stream) {
  g_err[0] = 0;
  if (src == nullptr || sink == nullptr) return fail(RP_ERR_INVALID_ARG, "src/sink is NULL");
  if (!aligned(src, 16) || !aligned(sink, 4)) return fail(RP_ERR_INVALID_ARG, "src must be 16-byte and sink 4-byte aligned");
  if (bytes == 0 || bytes % 16 != 0) return fail(RP_ERR_INVALID_ARG, "bytes must be a positive multiple of 16");
  hipError_t e = rp::launch_stream_read(src, bytes, sink, nontemporal != 0, stream);
  return e == hipSuccess ? RP_OK : hip_fail(e, "stream-read kernel launch");
}

}  // extern "C"

namespace rp {
rp_status set_error(rp_status st, const char* msg) {
  snprintf(g_err, sizeof(g_err), "%s", msg);
  return st;
}
void clear_error() { g_err[0] = 0; }
}  // namespace rp

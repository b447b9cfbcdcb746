// C-ABI of libsplash_attn: argument validation, workspace layout, the host
// mirror of the split planner, and the entry points declared in
// include/splash_attn.h.  No C++ exception crosses this boundary.
#include "splash_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <climits>
#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "splash_common.hpp"

using namespace splash;

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SPLASH_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  size_t off[6];  // header, units, indptr, split list, partial lse, partial out
  size_t total;
};

Layout layout_for(int64_t T, int32_t H, int64_t max_partials) {
  Layout L;
  size_t o = 0;
  L.off[0] = o; o = align_up(o + sizeof(int32_t) * kHeaderInts);
  L.off[1] = o; o = align_up(o + 16 * (size_t)(T + max_partials));
  L.off[2] = o; o = align_up(o + sizeof(int32_t) * (size_t)(T + 1));
  L.off[3] = o; o = align_up(o + sizeof(int4) * (size_t)(T > 0 ? T : 1));
  L.off[4] = o; o = align_up(o + sizeof(float) * (size_t)max_partials * H);
  L.off[5] = o; o = align_up(o + sizeof(float) * (size_t)max_partials * H * kDimV);
  L.total = o;
  return L;
}

// Largest partial capacity that fits in ws_bytes.
int64_t partials_for_bytes(int64_t T, int32_t H, size_t ws_bytes) {
  const Layout base = layout_for(T, H, 0);
  if (ws_bytes < base.total) return -1;
  const size_t per = 16 + sizeof(float) * (size_t)H * (1 + kDimV);
  int64_t mp = (int64_t)((ws_bytes - base.total) / per);
  if (mp > INT32_MAX / 2) mp = INT32_MAX / 2;
  while (mp > 0 && layout_for(T, H, mp).total > ws_bytes) --mp;
  return mp;
}

Workspace workspace_view(void* ws, int64_t T, int32_t H, int64_t max_partials) {
  const Layout L = layout_for(T, H, max_partials);
  char* base = static_cast<char*>(ws);
  Workspace w;
  w.header = reinterpret_cast<int32_t*>(base + L.off[0]);
  w.units = reinterpret_cast<int4*>(base + L.off[1]);
  w.indptr = reinterpret_cast<int32_t*>(base + L.off[2]);
  w.split_list = reinterpret_cast<int4*>(base + L.off[3]);
  w.part_lse = reinterpret_cast<float*>(base + L.off[4]);
  w.part_out = reinterpret_cast<float*>(base + L.off[5]);
  // the split partials in fp16 fill the first half of the region; the
  // quarter exponents follow them
  w.part_half = reinterpret_cast<uint16_t*>(base + L.off[5]);
  w.part_exp = reinterpret_cast<uint32_t*>(base + L.off[5] + sizeof(uint16_t) * (size_t)max_partials * H * kDimV);
  w.max_units = (int32_t)(T + max_partials);
  w.max_partials = (int32_t)max_partials;
  return w;
}

// Partial slots that the 1024-page unit cap alone can force.
int64_t forced_partials(int64_t T, int32_t max_pages_per_seq) {
  if (max_pages_per_seq <= kMaxUnitPages) return 0;
  return T * (int64_t)ceil_div(max_pages_per_seq, kMaxUnitPages);
}

int validate_desc(const splash_mla_desc* d, int32_t q_chunk) {
  if (!d) return fail(SPLASH_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->batch < 0) return fail(SPLASH_ERR_INVALID_ARGUMENT, "batch < 0");
  if (q_chunk < 1) return fail(SPLASH_ERR_INVALID_ARGUMENT, "q_chunk must be >= 1 (got %d)", q_chunk);
  if (d->dim_qk != kDimQK || d->dim_v != kDimV)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "dims must be qk=576, v=512 (got %d, %d)", d->dim_qk, d->dim_v);
  if (d->page_size != kPage) return fail(SPLASH_ERR_UNSUPPORTED, "page_size must be 64 (got %d)", d->page_size);
  if (d->num_heads < 16 || d->num_heads > kMaxHeads || d->num_heads % 16)
    return fail(SPLASH_ERR_UNSUPPORTED, "num_heads must be a multiple of 16 in [16,128] (got %d)", d->num_heads);
  if (d->kv_dtype != SPLASH_KV_BF16 && d->kv_dtype != SPLASH_KV_FP8_E4M3 && d->kv_dtype != SPLASH_KV_FP8_LATENT)
    return fail(SPLASH_ERR_UNSUPPORTED, "unknown kv_dtype %d", d->kv_dtype);
  if (d->kv_dtype == SPLASH_KV_FP8_E4M3 && !d->kv_scales)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "fp8 cache needs kv_scales");
  if (!(std::isfinite(d->softmax_scale) && d->softmax_scale > 0.f))
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  if (d->max_pages_per_seq < 1 || d->num_pages < 1)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "max_pages_per_seq and num_pages must be >= 1");
  if ((d->flags & SPLASH_FLAG_FORCE_SPLIT) && d->split_pages < 1)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "FORCE_SPLIT needs split_pages >= 1");
  if ((int64_t)d->batch * q_chunk > INT32_MAX / 2)
    return fail(SPLASH_ERR_UNSUPPORTED, "batch * q_chunk too large");
  return SPLASH_OK;
}

std::atomic<int32_t> g_workers[64];

int32_t device_workers() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
  int32_t w = g_workers[dev].load(std::memory_order_relaxed);
  if (w > 0) return w;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) return -1;
  g_workers[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Checks shared by plan / run / attend; fills the workspace view.
int prepare(const int32_t* seq_lens, int32_t q_chunk, const splash_mla_desc* d, void* workspace,
            size_t ws_bytes, Workspace* wv) {
  if (!seq_lens) return fail(SPLASH_ERR_INVALID_ARGUMENT, "seq_lens is NULL");
  if (!workspace) return fail(SPLASH_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SPLASH_ERR_MISALIGNED, "workspace not 16-byte aligned");
  if (d->kv_dtype == SPLASH_KV_FP8_E4M3 && !aligned16(d->kv_scales))
    return fail(SPLASH_ERR_MISALIGNED, "kv_scales not 16-byte aligned");
  const int64_t T = (int64_t)d->batch * q_chunk;
  const int64_t mp = partials_for_bytes(T, d->num_heads, ws_bytes);
  if (mp < 0)
    return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes is below the minimum %zu", ws_bytes,
                layout_for(T, d->num_heads, 0).total);
  if (mp < forced_partials(T, d->max_pages_per_seq))
    return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL,
                "histories longer than %d pages must be split: need room for %lld partials, have %lld",
                kMaxUnitPages, (long long)forced_partials(T, d->max_pages_per_seq), (long long)mp);
  *wv = workspace_view(workspace, T, d->num_heads, mp);
  return SPLASH_OK;
}

// One position shard of every request's history (splash_mla_attend_shard);
// all null for the whole history.
struct Shard {
  const int32_t* key_begin = nullptr;
  const int32_t* key_end = nullptr;
  int32_t num_shards = 0, shard = 0;
  // the top-k variant (splash_mla_attend_topk) travels the same way
  const int32_t* topk_idx = nullptr;
  const int32_t* topk_count = nullptr;
  int32_t topk = 0;
};

int check_device_data(const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens, int32_t q_chunk,
                      const splash_mla_desc* d, const Workspace& wv, hipStream_t s, const Shard& sh = Shard()) {
  int32_t* res = wv.header + kHdrDebug;
  const void* latent_kv = d->kv_dtype == SPLASH_KV_FP8_LATENT ? kv_pages : nullptr;
  hipError_t e = launch_check(block_table, seq_lens, latent_kv, sh.key_begin, sh.key_end, d->batch, q_chunk,
                              d->max_pages_per_seq, d->num_pages, res, s);
  if (e != hipSuccess) return hip_fail(e, "check launch");
  int32_t host = 0;
  e = hipMemcpyAsync(&host, res, sizeof host, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "check readback");
  if (host != INT32_MAX)
    return fail(SPLASH_ERR_INVALID_ARGUMENT,
                "request %d: seq_len < q_chunk, history longer than the block-table row, a block-table "
                "entry outside [0, num_pages), (shard) a key range that is not 0 <= begin <= end with begin "
                "a multiple of 64, or (latent-row cache) a tile scale that is not a positive power of two",
                host - 1);
  return SPLASH_OK;
}

int do_plan(const int32_t* seq_lens, int32_t q_chunk, const splash_mla_desc* d, const Workspace& wv,
            hipStream_t s, const Shard& sh = Shard()) {
  const int32_t G = device_workers();
  if (G < 1) return fail(SPLASH_ERR_HIP, "cannot query the device's compute units");
  PlanLaunch p;
  p.seq_lens = seq_lens;
  p.key_begin = sh.key_begin;
  p.key_end = sh.key_end;
  p.topk_count = sh.topk_count;
  p.unit_cap = sh.topk_idx ? kTopkUnitPages : kMaxUnitPages;
  p.B = d->batch;
  p.q_chunk = q_chunk;
  p.G = G;
  p.forced_chunk = (d->flags & SPLASH_FLAG_FORCE_SPLIT) ? d->split_pages : 0;
  p.ws = wv;
  hipError_t e = launch_plan(p, s);
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "plan launch");
}

int do_attend_units(const void* q, const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens,
                    int32_t q_chunk, void* out, float* lse, const splash_mla_desc* d, const Workspace& wv,
                    hipStream_t s, const Shard& sh = Shard()) {
  const int32_t G = device_workers();
  if (G < 1) return fail(SPLASH_ERR_HIP, "cannot query the device's compute units");
  AttendLaunch a;
  a.q = q;
  a.kv = kv_pages;
  a.kv_scales = d->kv_scales;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.key_begin = sh.key_begin;
  a.key_end = sh.key_end;
  a.topk_idx = sh.topk_idx;
  a.topk_count = sh.topk_count;
  a.topk = sh.topk;
  a.out = out;
  a.lse = lse;
  a.bt_stride = d->max_pages_per_seq;
  a.q_chunk = q_chunk;
  a.H = d->num_heads;
  a.kv_dtype = d->kv_dtype;
  a.B = d->batch;
  a.softmax_scale = d->softmax_scale;
  a.exact_qk = (d->flags & SPLASH_FLAG_EXACT_QK) ? 1 : 0;
  a.ws = wv;
  hipError_t e = launch_attend(a, G, s);
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "attend launch");
}

int do_combine_splits(int32_t q_chunk, void* out, float* lse, const splash_mla_desc* d, const Workspace& wv,
                      hipStream_t s, const Shard& sh = Shard()) {
  CombineLaunch c;
  c.partials = nullptr;
  c.partials_h = wv.part_half;
  c.part_exp = wv.part_exp;
  c.partial_lse = wv.part_lse;
  c.indptr = wv.indptr;
  c.item_list = wv.split_list;
  c.item_count = wv.header + kHdrSplitTiles;
  c.max_parts = wv.header + kHdrMaxParts;
  c.B = d->batch * q_chunk;
  c.q_chunk = 1;
  c.H = d->num_heads;
  c.out = out;
  c.out_lse = lse;
  // a shard or a top-k plan lists its tiles with no key, to be written empty
  c.write_empty = sh.key_end != nullptr || sh.topk_idx != nullptr;
  c.out_f32 = sh.key_end != nullptr;
  c.num_shards = sh.key_end ? sh.num_shards : 0;
  c.shard = sh.shard;
  c.tile_q = q_chunk;
  hipError_t e = launch_combine(c, s);
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "combine launch");
}

int do_run(const void* q, const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens,
           int32_t q_chunk, void* out, float* lse, const splash_mla_desc* d, const Workspace& wv, hipStream_t s) {
  int st = do_attend_units(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, d, wv, s);
  if (st != SPLASH_OK) return st;
  return do_combine_splits(q_chunk, out, lse, d, wv, s);
}

int check_tensors(const void* q, const void* kv_pages, const int32_t* block_table, void* out, const float* lse) {
  if (!q || !kv_pages || !block_table || !out)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "q, kv_pages, block_table and out must be non-NULL");
  if (!aligned16(q) || !aligned16(kv_pages) || !aligned16(out))
    return fail(SPLASH_ERR_MISALIGNED, "q, kv_pages and out must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(block_table) & 3u) || (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(SPLASH_ERR_MISALIGNED, "block_table and lse must be 4-byte aligned");
  return SPLASH_OK;
}

// ---- DOP regroup (sizes checked here; row_order is device data, a
// permutation of [0, num_rows) grouped by owner, and is not checked)
int dop_check(int64_t rows, int32_t hl, int32_t num_ranks, const void* const* ptrs, int nptr) {
  if (rows < 0 || hl < 1 || num_ranks < 1)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "need rows >= 0, heads_local >= 1, num_ranks >= 1");
  if (rows * hl * num_ranks * 72 >= INT32_MAX)
    return fail(SPLASH_ERR_UNSUPPORTED, "regroup too large (%lld rows)", (long long)rows);
  if (rows == 0) return SPLASH_OK;
  for (int i = 0; i < nptr; ++i) {
    if (!ptrs[i]) return fail(SPLASH_ERR_INVALID_ARGUMENT, "NULL buffer");
  }
  for (int i = 0; i < nptr; ++i) {
    if (i != 2 && !aligned16(ptrs[i]))  // slot 2, when used, is the int32 row order
      return fail(SPLASH_ERR_MISALIGNED, "regroup buffers must be 16-byte aligned");
  }
  return SPLASH_OK;
}

// Workspace of splash_mla_attend_noalloc: a device array of the library's
// own, one copy on every GPU the library runs on, held until the process
// ends.  In host code its name is only a stand-in, never a device address:
// the address comes from hipGetSymbolAddress, taken once per device with
// that device current, and only that address is passed on.
static __device__ __align__(256) uint8_t scratch[SPLASH_NOALLOC_SCRATCH_BYTES];
std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

int scratch_for_current_device(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(SPLASH_ERR_UNSUPPORTED, "device %d: the scratch table holds 64 devices", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(SPLASH_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SPLASH_OK;
}

}  // namespace

extern "C" {

size_t splash_mla_workspace_size(int32_t batch, int32_t q_chunk, int32_t num_heads, int32_t max_partials) {
  if (batch < 0 || q_chunk < 1 || num_heads < 1) return 0;
  if (max_partials <= 0) max_partials = SPLASH_DEFAULT_MAX_PARTIALS;
  return layout_for((int64_t)batch * q_chunk, num_heads, max_partials).total;
}

size_t splash_mla_workspace_offsets(int32_t batch, int32_t q_chunk, int32_t num_heads, int32_t max_partials,
                                    size_t* offsets) {
  if (batch < 0 || q_chunk < 1 || num_heads < 1) return 0;
  if (max_partials <= 0) max_partials = SPLASH_DEFAULT_MAX_PARTIALS;
  const Layout L = layout_for((int64_t)batch * q_chunk, num_heads, max_partials);
  if (offsets)
    for (int k = 0; k < 6; ++k) offsets[k] = L.off[k];
  return L.total;
}

int32_t splash_mla_max_units(int32_t batch, int32_t q_chunk, int32_t max_partials) {
  if (max_partials <= 0) max_partials = SPLASH_DEFAULT_MAX_PARTIALS;
  return (int32_t)((int64_t)batch * q_chunk + max_partials);
}

int32_t splash_device_workers(void) {
  const int32_t w = device_workers();
  return w < 1 ? 1 : w;
}

int splash_mla_plan(const int32_t* seq_lens, int32_t q_chunk, const splash_mla_desc* desc, void* workspace,
                    size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  return do_plan(seq_lens, q_chunk, desc, wv, static_cast<hipStream_t>(stream));
}

int splash_mla_run(const void* q, const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens,
                   int32_t q_chunk, void* out, float* lse, const splash_mla_desc* desc, void* workspace,
                   size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if ((st = check_tensors(q, kv_pages, block_table, out, lse)) != SPLASH_OK) return st;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->flags & SPLASH_FLAG_DEBUG_CHECK)
    if ((st = check_device_data(kv_pages, block_table, seq_lens, q_chunk, desc, wv, s)) != SPLASH_OK) return st;
  return do_run(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, desc, wv, s);
}

int splash_mla_attend_units(const void* q, const void* kv_pages, const int32_t* block_table,
                            const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                            const splash_mla_desc* desc, void* workspace, size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if ((st = check_tensors(q, kv_pages, block_table, out, lse)) != SPLASH_OK) return st;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  return do_attend_units(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, desc, wv,
                         static_cast<hipStream_t>(stream));
}

int splash_mla_combine_splits(int32_t q_chunk, void* out, float* lse, const splash_mla_desc* desc,
                              void* workspace, size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if (!out) return fail(SPLASH_ERR_INVALID_ARGUMENT, "out is NULL");
  if (!aligned16(out)) return fail(SPLASH_ERR_MISALIGNED, "out must be 16-byte aligned");
  if (!workspace) return fail(SPLASH_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (!aligned16(workspace)) return fail(SPLASH_ERR_MISALIGNED, "workspace not 16-byte aligned");
  const int64_t T = (int64_t)desc->batch * q_chunk;
  const int64_t mp = partials_for_bytes(T, desc->num_heads, ws_bytes);
  if (mp < 0) return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  const Workspace wv = workspace_view(workspace, T, desc->num_heads, mp);
  return do_combine_splits(q_chunk, out, lse, desc, wv, static_cast<hipStream_t>(stream));
}

int splash_mla_attend(const void* q, const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens,
                      int32_t q_chunk, void* out, float* lse, const splash_mla_desc* desc, void* workspace,
                      size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if ((st = check_tensors(q, kv_pages, block_table, out, lse)) != SPLASH_OK) return st;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->flags & SPLASH_FLAG_DEBUG_CHECK)
    if ((st = check_device_data(kv_pages, block_table, seq_lens, q_chunk, desc, wv, s)) != SPLASH_OK) return st;
  if ((st = do_plan(seq_lens, q_chunk, desc, wv, s)) != SPLASH_OK) return st;
  return do_run(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, desc, wv, s);
}

int splash_mla_attend_noalloc(const void* q, const void* kv_pages, const int32_t* block_table,
                              const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                              const splash_mla_desc* desc, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->flags & SPLASH_FLAG_DEBUG_CHECK)
    return fail(SPLASH_ERR_UNSUPPORTED,
                "splash_mla_attend_noalloc: DEBUG_CHECK reads its result back to the host; use splash_mla_attend");
  if (desc->batch == 0) return SPLASH_OK;
  const int64_t T = (int64_t)desc->batch * q_chunk;
  const size_t need = layout_for(T, desc->num_heads, forced_partials(T, desc->max_pages_per_seq)).total;
  if (need > SPLASH_NOALLOC_SCRATCH_BYTES)
    return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL,
                "splash_mla_attend_noalloc: this batch (%lld query rows, %d heads, up to %d pages per history) "
                "needs at least %zu bytes of workspace; the library's scratch holds %zu: use splash_mla_attend",
                (long long)T, desc->num_heads, desc->max_pages_per_seq, need, (size_t)SPLASH_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_for_current_device(&ws)) != SPLASH_OK) return st;
  return splash_mla_attend(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, desc, ws,
                           SPLASH_NOALLOC_SCRATCH_BYTES, stream);
}

int splash_mla_attend_topk(const void* q, const void* kv_pages, const int32_t* block_table,
                           const int32_t* seq_lens, int32_t q_chunk, const int32_t* topk_idx,
                           const int32_t* topk_count, int32_t topk, void* out, float* lse,
                           const splash_mla_desc* desc, void* workspace, size_t ws_bytes, void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if (!topk_idx || !topk_count) return fail(SPLASH_ERR_INVALID_ARGUMENT, "topk_idx and topk_count must be non-NULL");
  if (topk < 1 || topk > (1 << 24)) return fail(SPLASH_ERR_INVALID_ARGUMENT, "topk must be in [1, 2^24] (got %d)", topk);
  if ((desc->flags & SPLASH_FLAG_FORCE_SPLIT) && desc->split_pages > kTopkUnitPages)
    return fail(SPLASH_ERR_UNSUPPORTED, "a top-k unit holds at most %d x 64 entries", kTopkUnitPages);
  if ((st = check_tensors(q, kv_pages, block_table, out, lse)) != SPLASH_OK) return st;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  const int64_t N = (int64_t)desc->batch * q_chunk;
  const int64_t groups = ceil_div(topk, kPage);
  const int64_t need = groups > kTopkUnitPages ? N * ceil_div((int32_t)groups, kTopkUnitPages) : 0;
  if (wv.max_partials < need)
    return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL, "lists longer than %d entries are split: need %lld partial slots, have %d",
                kTopkUnitPages * kPage, (long long)need, wv.max_partials);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (desc->flags & SPLASH_FLAG_DEBUG_CHECK) {
    int32_t* res = wv.header + kHdrDebug;
    const void* latent_kv = desc->kv_dtype == SPLASH_KV_FP8_LATENT ? kv_pages : nullptr;
    hipError_t e = launch_topk_check(block_table, seq_lens, topk_idx, topk_count, (int32_t)N, q_chunk, topk,
                                     desc->max_pages_per_seq, desc->num_pages, latent_kv, res, s);
    if (e != hipSuccess) return hip_fail(e, "check launch");
    int32_t host = 0;
    e = hipMemcpyAsync(&host, res, sizeof host, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "check readback");
    if (host != INT32_MAX)
      return fail(SPLASH_ERR_INVALID_ARGUMENT,
                  "row %d: count outside [0, topk], a position outside the row's visible prefix, its block-table "
                  "entry outside [0, num_pages), or (latent-row cache) a listed row's tile scale that is not a "
                  "positive power of two",
                  host - 1);
  }
  Shard sh;
  sh.topk_idx = topk_idx;
  sh.topk_count = topk_count;
  sh.topk = topk;
  if ((st = do_plan(seq_lens, q_chunk, desc, wv, s, sh)) != SPLASH_OK) return st;
  if ((st = do_attend_units(q, kv_pages, block_table, seq_lens, q_chunk, out, lse, desc, wv, s, sh)) != SPLASH_OK)
    return st;
  return do_combine_splits(q_chunk, out, lse, desc, wv, s, sh);
}

int splash_mla_attend_shard(const void* q, const void* kv_pages, const int32_t* block_table,
                            const int32_t* seq_lens, int32_t q_chunk, const int32_t* key_begin,
                            const int32_t* key_end, int32_t num_shards, int32_t shard, float* part_out,
                            float* part_lse, const splash_mla_desc* desc, void* workspace, size_t ws_bytes,
                            void* stream) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if (!key_begin || !key_end || !part_lse)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "key_begin, key_end and part_lse must be non-NULL");
  if (num_shards < 1 || shard < 0 || shard >= num_shards)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "need 0 <= shard < num_shards (got %d of %d)", shard, num_shards);
  if (desc->flags & SPLASH_FLAG_FORCE_SPLIT)
    return fail(SPLASH_ERR_UNSUPPORTED, "FORCE_SPLIT does not apply to a shard");
  if ((st = check_tensors(q, kv_pages, block_table, part_out, part_lse)) != SPLASH_OK) return st;
  Workspace wv;
  if ((st = prepare(seq_lens, q_chunk, desc, workspace, ws_bytes, &wv)) != SPLASH_OK) return st;
  const int64_t T = (int64_t)desc->batch * q_chunk;
  if (wv.max_partials < T)
    return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL,
                "a shard needs a partial slot for every query row: %lld, the workspace has %d", (long long)T,
                wv.max_partials);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Shard sh;
  sh.key_begin = key_begin;
  sh.key_end = key_end;
  sh.num_shards = num_shards;
  sh.shard = shard;
  if (desc->flags & SPLASH_FLAG_DEBUG_CHECK)
    if ((st = check_device_data(kv_pages, block_table, seq_lens, q_chunk, desc, wv, s, sh)) != SPLASH_OK) return st;
  if ((st = do_plan(seq_lens, q_chunk, desc, wv, s, sh)) != SPLASH_OK) return st;
  if ((st = do_attend_units(q, kv_pages, block_table, seq_lens, q_chunk, part_out, part_lse, desc, wv, s, sh)) !=
      SPLASH_OK)
    return st;
  return do_combine_splits(q_chunk, part_out, part_lse, desc, wv, s, sh);
}

int splash_mla_combine(const float* partials, const float* partial_lse, const int32_t* split_indptr, int32_t batch,
                       int32_t q_chunk, int32_t num_heads, void* out, float* out_lse, void* stream) {
  if (batch < 0 || q_chunk < 1 || num_heads < 1)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "batch >= 0, q_chunk >= 1 and num_heads >= 1 required");
  if (batch == 0) return SPLASH_OK;
  if (!partials || !partial_lse || !split_indptr || !out)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "partials, partial_lse, split_indptr and out must be non-NULL");
  if (!aligned16(partials) || !aligned16(out))
    return fail(SPLASH_ERR_MISALIGNED, "partials and out must be 16-byte aligned");
  CombineLaunch c;
  c.partials = partials;
  c.partials_h = nullptr;
  c.part_exp = nullptr;
  c.partial_lse = partial_lse;
  c.indptr = split_indptr;
  c.item_list = nullptr;
  c.item_count = nullptr;
  c.max_parts = nullptr;
  c.B = batch;
  c.q_chunk = q_chunk;
  c.H = num_heads;
  c.out = out;
  c.out_lse = out_lse;
  c.write_empty = true;
  c.out_f32 = false;
  c.num_shards = 0;
  c.shard = 0;
  c.tile_q = 1;
  hipError_t e = launch_combine(c, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "combine launch");
}

int splash_mla_debug_gather(const void* kv_pages, const int32_t* block_table, const int32_t* seq_lens,
                            const splash_mla_desc* desc, void* dense_out, void* stream) {
  int st = validate_desc(desc, 1);
  if (st != SPLASH_OK) return st;
  if (desc->batch == 0) return SPLASH_OK;
  if (!kv_pages || !block_table || !seq_lens || !dense_out)
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "kv_pages, block_table, seq_lens and dense_out must be non-NULL");
  if (!aligned16(kv_pages) || !aligned16(dense_out))
    return fail(SPLASH_ERR_MISALIGNED, "kv_pages and dense_out must be 16-byte aligned");
  const int32_t row_bytes = desc->kv_dtype == SPLASH_KV_FP8_LATENT ? kLatentRowBytes
                            : desc->kv_dtype == SPLASH_KV_FP8_E4M3 ? kDimQK : 2 * kDimQK;
  hipError_t e = launch_gather(kv_pages, block_table, seq_lens, desc->batch, desc->max_pages_per_seq, row_bytes,
                               dense_out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "gather launch");
}

int splash_mla_plan_host(const int32_t* seq_lens_host, int32_t q_chunk, const splash_mla_desc* desc,
                         int32_t num_workers, int32_t max_partials, int32_t* units_out, int32_t max_units,
                         int32_t* indptr_out, int32_t* stats_out, int32_t* worker_start_out) {
  int st = validate_desc(desc, q_chunk);
  if (st != SPLASH_OK) return st;
  if (num_workers < 1) return fail(SPLASH_ERR_INVALID_ARGUMENT, "num_workers must be >= 1");
  const int32_t B = desc->batch, T = B * q_chunk;
  if (B > 0 && (!seq_lens_host || !units_out || !indptr_out || !stats_out))
    return fail(SPLASH_ERR_INVALID_ARGUMENT, "NULL host buffer");
  if (max_partials <= 0) max_partials = SPLASH_DEFAULT_MAX_PARTIALS;
  const int32_t G = num_workers;
  std::vector<int32_t> P((size_t)std::max(T, 1));
  int64_t total = 0;
  int32_t mx = 0;
  for (int32_t t = 0; t < T; ++t) {
    const int32_t b = t / q_chunk, i = t - b * q_chunk;
    const int32_t L = tile_keys(seq_lens_host[b], q_chunk, i);
    P[t] = L > 0 ? ceil_div(L, kPage) : 0;
    total += P[t];
    mx = std::max(mx, P[t]);
  }
  const int32_t max_pages = mx > 0 ? mx : 1;
  const int32_t cap_units = std::min<int64_t>(max_units, (int64_t)T + max_partials);
  auto evaluate = [&](int32_t c, int64_t* cost) {
    int64_t W = 0, S = 0;
    for (int32_t t = 0; t < T; ++t) {
      const int32_t n = P[t] > 0 ? ceil_div(P[t], c) : 0;
      W += n;
      S += n > 1 ? n : 0;
    }
    const bool ok = S <= max_partials && W <= (int64_t)T + max_partials;
    *cost = ok ? plan_cost(c, W, S, total, max_pages, G, kPlanCosts) : INT64_MAX;
  };
  int32_t best_c = 0;
  int64_t best = INT64_MAX;
  for (int k = 0; k < kNumCandidates; ++k) {
    const int32_t c = plan_candidate(k, max_pages);
    int64_t cost;
    evaluate(c, &cost);
    if (k == 0 || cost < best) {
      best = cost;
      best_c = c;
    }
  }
  const bool forced = (desc->flags & SPLASH_FLAG_FORCE_SPLIT) != 0;
  if (forced) {
    const int32_t c = std::min(desc->split_pages, (int32_t)kMaxUnitPages);
    int64_t cost;
    evaluate(c, &cost);
    if (cost != INT64_MAX) best_c = c;
  }
  const int32_t c = best_c;
  // the fold plan: ranks by pages (longest first, ties by tile), then the
  // cheapest cap, largest on ties
  bool fold = !forced && fold_applicable(T, G, kMaxWorkers, max_pages, total, best, kPlanCosts);
  int32_t cap = 0, nl = 0;
  std::vector<int32_t> q((size_t)std::max(G, 1), 0), rank_tile((size_t)std::max(T, 1));
  if (fold) {
    for (int32_t t = 0; t < T; ++t) rank_tile[t] = t;
    std::stable_sort(rank_tile.begin(), rank_tile.begin() + T, [&](int32_t a, int32_t b) { return P[a] > P[b]; });
    for (int32_t r = 0; r < T; ++r) q[r] = P[rank_tile[r]];
    int64_t fbest = INT64_MAX;
    for (int32_t C = q[0] - 1; C >= 1; --C) {
      int32_t n;
      const int64_t cost = fold_cost(C, q, G, max_partials, kPlanCosts, &n);
      if (cost < fbest) {
        fbest = cost;
        cap = C;
      }
    }
    fold = fbest != INT64_MAX && fbest < best;
    if (fold) fold_cost(cap, q, G, max_partials, kPlanCosts, &nl);
  }
  int32_t nu = 0, ns = 0;
  if (fold) {
    // partial slots in tile order; units worker by worker
    for (int32_t t = 0; t < T; ++t) {
      indptr_out[t] = ns;
      ns += P[t] > cap ? 2 : 0;
    }
    indptr_out[T] = ns;
    if ((int64_t)T + nl > cap_units) return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL, "more units than max_units");
    for (int32_t r = 0; r < G; ++r) {
      if (worker_start_out) worker_start_out[r] = nu;
      if (r < T && q[r] > 0) {
        const int32_t t = rank_tile[r];
        int32_t* u = units_out + 4 * (size_t)nu++;
        u[0] = t;
        u[1] = 0;
        u[2] = r < nl ? cap : q[r];
        u[3] = r < nl ? indptr_out[t] : -1;
      }
      if (r >= G - nl) {
        const int32_t j = G - 1 - r, t = rank_tile[j];
        int32_t* u = units_out + 4 * (size_t)nu++;
        u[0] = t;
        u[1] = cap;
        u[2] = q[j];
        u[3] = indptr_out[t] + 1;
      }
    }
    if (worker_start_out) worker_start_out[G] = nu;
  } else {
    for (int32_t t = 0; t < T; ++t) {
      const int32_t n = P[t] > 0 ? ceil_div(P[t], c) : 0;
      indptr_out[t] = ns;
      for (int32_t u = 0; u < n; ++u) {
        if (nu >= cap_units) return fail(SPLASH_ERR_WORKSPACE_TOO_SMALL, "more units than max_units");
        int32_t* r = units_out + 4 * (size_t)nu++;
        r[0] = t;
        r[1] = unit_begin(P[t], n, u);
        r[2] = unit_begin(P[t], n, u + 1);
        r[3] = n > 1 ? ns + u : -1;
      }
      ns += n > 1 ? n : 0;
    }
    if (T >= 0 && indptr_out) indptr_out[T] = ns;
    if (T <= kPlanLdsTiles && nu > G) {
      // the device queue order: longest unit first (equal lengths in tile
      // order here; the device leaves their order open).  With query chunks
      // (up to kMaxWorkers requests), whole requests instead, keyed by their
      // longest unit (ties in request order here), each request's units
      // unit index major (the rows of one page range side by side).
      // rows[i][4] is the unit's index inside its tile.
      std::vector<std::array<int32_t, 5>> rows((size_t)nu);
      for (int32_t i = 0; i < nu; ++i) {
        for (int j = 0; j < 4; ++j) rows[i][j] = units_out[4 * (size_t)i + j];
        rows[i][4] = (i > 0 && rows[i - 1][0] == rows[i][0]) ? rows[i - 1][4] + 1 : 0;
      }
      std::vector<int32_t> rkey((size_t)std::max(B, 1), 0);
      const bool grouped = q_chunk > 1 && B <= kMaxWorkers;
      if (grouped)
        for (const auto& r : rows) rkey[r[0] / q_chunk] = std::max(rkey[r[0] / q_chunk], r[2] - r[1]);
      std::stable_sort(rows.begin(), rows.end(),
                       [&](const std::array<int32_t, 5>& a, const std::array<int32_t, 5>& b) {
                         if (grouped) {
                           const int32_t ra = a[0] / q_chunk, rb = b[0] / q_chunk;
                           if (rkey[ra] != rkey[rb]) return rkey[ra] > rkey[rb];
                           if (ra != rb) return ra < rb;
                           if (a[4] != b[4]) return a[4] < b[4];
                           return a[0] < b[0];
                         }
                         return a[2] - a[1] > b[2] - b[1];
                       });
      for (int32_t i = 0; i < nu; ++i)
        for (int j = 0; j < 4; ++j) units_out[4 * (size_t)i + j] = rows[i][j];
    }
  }
  if (stats_out) {
    stats_out[0] = nu;
    stats_out[1] = ns;
    stats_out[2] = fold ? 0 : c;
    stats_out[3] = total > INT32_MAX ? INT32_MAX : (int32_t)total;
    stats_out[4] = fold ? G : 0;
    stats_out[5] = fold ? cap : 0;
    stats_out[6] = fold ? (nl > 0 ? 2 : 1) : (max_pages + c - 1) / c;
  }
  return SPLASH_OK;
}

int splash_dop_pack_q(const void* q_nope, const void* q_rope, const int32_t* row_order, int32_t num_rows,
                      int32_t heads_local, void* send, void* stream) {
  const void* ptrs[4] = {q_nope, q_rope, row_order, send};
  int st = dop_check(num_rows, heads_local, 1, ptrs, 4);
  if (st != SPLASH_OK || num_rows == 0) return st;
  hipError_t e = launch_dop_pack_q(q_nope, q_rope, row_order, num_rows, heads_local, send,
                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "dop pack_q launch");
}

int splash_dop_unpack_q(const void* recv, int32_t num_ranks, int32_t owner_rows, int32_t heads_local, void* q_owner,
                        void* stream) {
  const void* ptrs[2] = {recv, q_owner};
  int st = dop_check(owner_rows, heads_local, num_ranks, ptrs, 2);
  if (st != SPLASH_OK || owner_rows == 0) return st;
  hipError_t e = launch_dop_unpack_q(recv, num_ranks, owner_rows, heads_local, q_owner,
                                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "dop unpack_q launch");
}

int splash_dop_pack_out(const void* out_owner, int32_t num_ranks, int32_t owner_rows, int32_t heads_local, void* send,
                        void* stream) {
  const void* ptrs[2] = {out_owner, send};
  int st = dop_check(owner_rows, heads_local, num_ranks, ptrs, 2);
  if (st != SPLASH_OK || owner_rows == 0) return st;
  hipError_t e = launch_dop_pack_out(out_owner, num_ranks, owner_rows, heads_local, send,
                                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "dop pack_out launch");
}

int splash_dop_unpack_out(const void* recv, const int32_t* row_order, int32_t num_rows, int32_t heads_local, void* out,
                          void* stream) {
  const void* ptrs[4] = {recv, out, row_order, out};
  int st = dop_check(num_rows, heads_local, 1, ptrs, 4);
  if (st != SPLASH_OK || num_rows == 0) return st;
  hipError_t e = launch_dop_unpack_out(recv, row_order, num_rows, heads_local, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SPLASH_OK : hip_fail(e, "dop unpack_out launch");
}

const char* splash_status_string(int status) {
  switch (status) {
    case SPLASH_OK: return "ok";
    case SPLASH_ERR_INVALID_ARGUMENT: return "invalid argument";
    case SPLASH_ERR_UNSUPPORTED: return "unsupported";
    case SPLASH_ERR_MISALIGNED: return "misaligned pointer";
    case SPLASH_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case SPLASH_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* splash_last_error(void) { return g_last_error.c_str(); }

const char* splash_version(void) { return "libsplash_attn 0.1.0 (gfx950)"; }

}  // extern "C"

// Internal launch interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "splash_common.hpp"

namespace splash {

struct Workspace {
  int32_t* header;      // kHeaderInts ints
  int4* units;          // [max_units]
  int32_t* indptr;      // [T + 1]
  int4* split_list;     // [T] {tile, first partial slot, parts, 0} of the tiles with partials (count in the header)
  float* part_lse;      // [max_partials, H]
  float* part_out;      // region of [max_partials, H, 512] floats, which holds the split partials as
  uint16_t* part_half;  //   fp16 [max_partials, H, 512] (its first half), each (slot, head) 128-column
  uint32_t* part_exp;   //   quarter q scaled by 2^-e with e = byte q of part_exp[slot * H + head]
  int32_t max_units;
  int32_t max_partials;
};

// Header slots.
enum HeaderSlot : int {
  kHdrGrab = 0,        // unused (written as 0)
  kHdrUnits = 1,       // number of work units
  kHdrPartials = 2,    // partial slots used
  kHdrChunk = 3,       // pages per unit
  kHdrDebug = 4,       // device-data check result (0 ok, else first failing item + 1)
  kHdrDone = 5,        // unused (written as 0)
  kHdrSplitTiles = 6,  // number of tiles with partials
  kHdrTotalPages = 7,
  kHdrMaxParts = 8,    // upper bound on the parts of any split tile
  kHdrSchedule = 9,    // 0: the queue (longest unit first), dealt to the G workers in a snake;
                       // G > 0: fold plan for G workers, worker g runs units [table[g], table[g + 1])
  kHdrFoldCap = 10,    // fold plan: pages a long tile keeps (its tail goes to a partner worker)
  kHdrWorkerTable = 64,  // fold plan: first unit of each worker, G + 1 entries
};

struct PlanLaunch {
  const int32_t* seq_lens;
  const int32_t* key_begin;  // shard: request b's keys [key_begin[b], key_end[b]) (nullptr: whole history)
  const int32_t* key_end;
  const int32_t* topk_count;  // top-k variant: row n attends its first topk_count[n] selected tokens
  int32_t B, q_chunk, G, forced_chunk;
  int32_t unit_cap;           // largest unit in pages (kMaxUnitPages, or kTopkUnitPages for top-k)
  Workspace ws;
};

struct AttendLaunch {
  const void* q;
  const void* kv;
  const float* kv_scales;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* key_begin;  // shard (see PlanLaunch): unit pages count from key_begin[b] / 64
  const int32_t* key_end;
  const int32_t* topk_idx;    // top-k variant: [N, topk] selected token positions of each row
  const int32_t* topk_count;  // [N] how many of them are used
  int32_t topk;
  void* out;
  float* lse;
  int32_t bt_stride, q_chunk, H, kv_dtype, B;
  float softmax_scale;
  int32_t exact_qk;  // fp8 caches: QK with K converted to bf16 (fp32-exact products), not on the fp8 pipe
  Workspace ws;
};

struct CombineLaunch {
  const float* partials;      // fp32 partials (the standalone merge), or
  const uint16_t* partials_h; // the attend kernel's fp16 partials with their quarter exponents
  const uint32_t* part_exp;
  const float* partial_lse;
  const int32_t* indptr;     // [B + 1] partial-slot offsets (per request or per tile)
  const int4* item_list;     // optional {request, first slot, parts, 0} records to process (count from
                             // *item_count); without it every request, with its range from indptr
  const int32_t* item_count;
  const int32_t* max_parts;  // optional bound on the parts of every listed item
  int32_t B, q_chunk, H;
  void* out;
  float* out_lse;
  bool write_empty;          // requests without partials get out = 0, lse = -inf
  bool out_f32;              // out is fp32 (a shard's partial result) instead of bf16
  int32_t num_shards, shard, tile_q;  // num_shards > 0: output row r = b' * tile_q + i goes to row
                                      // (b' * num_shards + shard) * tile_q + i
};

hipError_t launch_plan(const PlanLaunch& p, hipStream_t s);
hipError_t launch_attend(const AttendLaunch& p, int32_t workers, hipStream_t s);
hipError_t launch_combine(const CombineLaunch& p, hipStream_t s);
hipError_t launch_gather(const void* kv, const int32_t* bt, const int32_t* seq_lens, int32_t B,
                         int32_t bt_stride, int32_t row_bytes, void* dense, hipStream_t s);
hipError_t launch_topk_check(const int32_t* bt, const int32_t* seq_lens, const int32_t* idx, const int32_t* count,
                             int32_t N, int32_t q_chunk, int32_t topk, int32_t bt_stride, int32_t num_pages,
                             const void* latent_kv, int32_t* result, hipStream_t s);
hipError_t launch_dop_pack_q(const void* q_nope, const void* q_rope, const int32_t* order, int32_t n, int32_t hl,
                             void* send, hipStream_t s);
hipError_t launch_dop_unpack_q(const void* recv, int32_t T, int32_t n, int32_t hl, void* q_owner, hipStream_t s);
hipError_t launch_dop_pack_out(const void* out_owner, int32_t T, int32_t n, int32_t hl, void* send, hipStream_t s);
hipError_t launch_dop_unpack_out(const void* recv, const int32_t* order, int32_t n, int32_t hl, void* out,
                                 hipStream_t s);
hipError_t launch_check(const int32_t* bt, const int32_t* seq_lens, const void* latent_kv, const int32_t* key_begin,
                        const int32_t* key_end, int32_t B, int32_t q_chunk, int32_t bt_stride, int32_t num_pages,
                        int32_t* result, hipStream_t s);

}  // namespace splash

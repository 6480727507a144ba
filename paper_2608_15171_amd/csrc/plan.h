// Work list of one mixed step: what each workgroup of the packed attention
// launch computes, and how split rows are merged afterwards.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "ppas.h"

namespace ppas {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kGroup = 8;          // query heads per KV head
// positions per prefill tile (x 8 heads): 16 for the four-wave kernel, 32 for
// the eight-wave one; each plan uses one of them
constexpr int kTilePosSmall = 16;
constexpr int kTilePosLarge = 32;
constexpr int kPrefillBlock = 64;  // keys per staged K/V block of a prefill tile
constexpr int kDecodeBlock = 32;   // keys per block of a decode wave
constexpr int kDecodeMaxKeys = 16384;  // longest key range of one decode item
constexpr int kKindPrefill = 0;
constexpr int kKindDecode = 1;

// One workgroup's job. A prefill tile covers npos consecutive positions of one
// request (rows row0..row0+npos-1 of the step, positions pos0..pos0+npos-1) for
// the 8 query heads of KV head kvh, over keys [key_lo, key_hi). A decode item is
// the same with npos == 1. part < 0: write bf16 output; else write fp32 partial
// (max, sum, unnormalised accumulator) for local row r = pos*8 + head at slot part + r.
struct WorkItem {
  int32_t seq, kvh, row0, pos0;
  int32_t npos_kind;               // npos | kind << 16
  int32_t key_lo, key_hi, part;
};
static_assert(sizeof(WorkItem) == 32, "WorkItem is 32 bytes");

// Rows split over nsplit items: split s of local row r sits at slot part + s*npos*8 + r.
struct CombineItem {
  int32_t row0, kvh, npos, nsplit, part, pad0, pad1, pad2;
};
static_assert(sizeof(CombineItem) == 32, "CombineItem is 32 bytes");

// One workgroup of the page-write kernels: the new rows of request `seq` that fall
// in its logical page `lpage` (positions lpage*16.. of the request), for every KV
// head. The request's rows are query_start..query_start+n_query-1 at positions
// cached_len..cached_len+n_query-1.
struct AppendItem {
  int32_t seq, lpage, cached_len, n_query, query_start, pad0, pad1, pad2;
};
static_assert(sizeof(AppendItem) == 32, "AppendItem is 32 bytes");

// Per-call planning choices; zero selects the automatic one.
struct PlanOpts {
  int32_t prefill_split = 0;       // >0: keys per prefill work item at most (rounded up to 64)
  int32_t decode_split = 0;        // >0: keys per decode work item at most (rounded up to 32)
  int32_t tile_pos = 0;            // 16 or 32 forces the prefill tile shape
};

struct Plan {
  int tile_pos = kTilePosSmall;    // prefill tile positions, selects the kernel shape
  std::vector<WorkItem> items;     // in launch order
  std::vector<CombineItem> combine;
  int64_t part_slots = 0;
  // work list as the kernels read it (bytes): items from 0, combine items at off_combine
  size_t off_combine = 0, list_bytes = 0;
  // caller workspace layout (bytes): the split partials (max, sum) then accumulators
  size_t off_ml = 0, off_acc = 0, total = 0;
};

ppas_status validate(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                     const int32_t* bt_host, int32_t bt_stride, bool check_overlap);

// Builds the plan for a device with num_cus compute units. The step must already be valid.
void make_plan(const ppas_shape& shape, const ppas_seq* seqs, int32_t n_seqs, int num_cus, const PlanOpts& opts,
               Plan& plan);

// The page-write work of a valid step: one item per (request, touched logical page).
void make_append_items(const ppas_seq* seqs, int32_t n_seqs, std::vector<AppendItem>& items);

}  // namespace ppas

// Device work-list records shared by the planner (host) and the kernels.
// Plain 16/32-byte PODs so one host buffer can be copied to the device as is.
#pragma once
#include <cstdint>

namespace spanq {

constexpr int kPage = 16;  // tokens per page on device pools

// One page of a query's key/value list.  Key slot s of the page sits at position
// pos0 + s in the frame of the rows reading it; the page stores keys rotated at
// position (pos0 - delta) + s, so a reader rotates them by `delta` more.
struct KvPage {
  int32_t page_id;
  int32_t n_valid;  // filled slots (a span's last page may be partial)
  int32_t pos0;
  int32_t delta;
};

// A key tile of the MFMA kernels: the four pages kv[4i .. 4i + 3] of a key list
// padded to whole tiles, reduced to what the kernels read.  One 32-byte record per
// tile, so one 64-byte scalar cache line serves two tiles (four 16-byte page
// records would take a line per tile).
struct TileRec {
  int32_t page_id[4];
  int32_t pos0;   // position of key 0 (all four pages come from one span)
  int32_t nk;     // real keys: the n_valid of the four pages summed
  int32_t delta;  // reposition delta, one per tile
  int32_t pad;
};

// One page to fill from caller rows: slots 0..n_valid-1 come from rows
// src_row.., keys rotated at positions pos0...
struct NewPage {
  int32_t page_id;
  int32_t n_valid;
  int32_t src_row;
  int32_t pos0;
};

// One repositioned copy (materialised repositioning): the keys of page src_page,
// stored at positions p.., are written to page dst_page rotated to positions
// p + delta..; the values are copied as they are.
struct MovePage {
  int32_t src_page;
  int32_t dst_page;
  int32_t delta;
  int32_t n_valid;
};

// Decoded tokens to write into a page: slots slot0 .. slot0 + n - 1 from caller rows
// src_row .., keys rotated at positions pos0 ..; the page's other slots are left as
// they are.
struct SlotWrite {
  int32_t page_id;
  int32_t slot0;
  int32_t n;
  int32_t src_row;
  int32_t pos0;
  int32_t pad[3];
};

// A tile of up to BM consecutive query rows of one span, against the key pages
// kv[kv_begin, kv_end).  part < 0: write the normalised output; else write the
// partial of one KV split (O / l, m, l) into partial slot `part`.  With
// kTwoKeyGroups (MFMA kernel, rows <= 32, four query heads per kv head) the two
// 32-row wave groups of the work-group take alternate key tiles instead of two
// row blocks, and write partial slots part and part + 1.
// Cross tiles also name the cross-segment pages of their key range (flags >> 8 of
// them, from entry w_first of the plan's cross page writes), which the MFMA cross
// kernel writes itself before reading them when the launch asks it to.
constexpr int32_t kTwoKeyGroups = 1;
constexpr int kWriteShift = 8;
struct WorkTile {
  int32_t q_row0;
  int32_t n_rows;
  int32_t q_pos0;
  int32_t kv_begin;
  int32_t kv_end;
  int32_t part;
  int32_t flags;
  int32_t w_first;
};

// Merge partial slots part0..part0+n_parts-1 into output rows q_row0...
struct CombineTile {
  int32_t q_row0;
  int32_t n_rows;
  int32_t part0;
  int32_t n_parts;
};

}  // namespace spanq

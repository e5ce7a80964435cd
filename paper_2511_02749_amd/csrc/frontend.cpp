// Parser of serialized span queries (server side of the front-end).
//
// A client serializes the optimized span query G(Cross(prefix.., Plus(F1..Fn),
// cross..)) with special tokens (section 5.2 and Def. 4; block alignment of section
// 5.3): OPEN "(" starts the commutative join's first child, SEP ")(" each next one,
// CLOSE ")" ends the join and is followed by the position of its OPEN (the variant
// of the paper that spares the server a parsing stack).  Every special token starts
// a block; PAD tokens fill the end of the block before it.  This parser recovers the
// spans the planner takes: the prefix before the join, each child, the cross segment
// after it.  Special and pad tokens are not part of any span (the library keeps no
// pad tokens in attention).
#include <cstdint>
#include <string>

#include "../../include/spanq.h"
#include "capi_internal.h"

namespace {

int bad(const std::string& what, int64_t at) {
  return spanq::report(SPAN_EINVAL, ("span_parse_serialized: " + what + " at token " + std::to_string(at)).c_str());
}

}  // namespace

extern "C" int span_parse_serialized(const int32_t* tok, int64_t n, int32_t block, const int32_t special[4],
                                     span_range* frags, int32_t cap, int32_t* n_frags, span_range* prefix,
                                     span_range* cross) {
  if ((!tok && n > 0) || n < 0 || block < 1 || !special || !n_frags || !prefix || !cross || cap < 0 ||
      (cap > 0 && !frags))
    return spanq::report(SPAN_EINVAL, "span_parse_serialized: bad argument");
  const int32_t PAD = special[0], OPEN = special[1], SEP = special[2], CLOSE = special[3];
  auto is_special = [&](int32_t t) { return t == PAD || t == OPEN || t == SEP || t == CLOSE; };
  // content [b, e) followed by pads up to e_pad: pads only after the content
  auto content = [&](int64_t b, int64_t e, const char* what, span_range* out) -> int {
    int64_t c = e;
    while (c > b && tok[c - 1] == PAD) --c;
    for (int64_t i = b; i < c; ++i)
      if (is_special(tok[i])) return bad(std::string("special token inside the ") + what, i);
    out->begin = b;
    out->n = c - b;
    return SPAN_OK;
  };
  int64_t open_at = -1;
  for (int64_t i = 0; i < n; ++i)
    if (tok[i] == OPEN) {
      open_at = i;
      break;
    }
  *n_frags = 0;
  if (open_at < 0) {  // no commutative join: everything is the cross segment
    prefix->begin = 0;
    prefix->n = 0;
    for (int64_t i = 0; i < n; ++i)
      if (is_special(tok[i])) return bad("special token without an open join", i);
    cross->begin = 0;
    cross->n = n;
    return SPAN_OK;
  }
  if (open_at % block != 0) return bad("OPEN not at a block start", open_at);
  int rc = content(0, open_at, "prefix", prefix);
  if (rc) return rc;
  int64_t start = open_at;  // position of the special token opening the current child
  int32_t k = 0;
  for (;;) {
    int64_t q = start + 1;
    while (q < n && !(tok[q] == SEP || tok[q] == CLOSE || tok[q] == OPEN)) ++q;
    if (q >= n) return bad("join not closed", start);
    if (tok[q] == OPEN) return bad("nested join (one commutative join per query)", q);
    if (q % block != 0) return bad("special token not at a block start", q);
    span_range r{};
    rc = content(start + 1, q, "fragment", &r);
    if (rc) return rc;
    if (k < cap) frags[k] = r;
    ++k;
    if (tok[q] == CLOSE) {
      if (q + 1 >= n) return bad("CLOSE without the position of its OPEN", q);
      if (tok[q + 1] != open_at) return bad("CLOSE points to " + std::to_string(tok[q + 1]) + ", not to its OPEN", q);
      for (int64_t i = q + 2; i < n; ++i)
        if (is_special(tok[i])) return bad("special token after the join", i);
      cross->begin = q + 2;
      cross->n = n - (q + 2);
      break;
    }
    start = q;
  }
  *n_frags = k;
  return SPAN_OK;
}

// Host-only check of the forward launch schedule (append_fwd_schedule in
// paper_2502_06155_amd/csrc/tile_attn_host.cpp), linked against the built library and
// run by tests/test_schedule.py: for each shape, every (unit, kept tile) is covered
// exactly once by the whole units and the parts of the schedule, every unit with rows
// runs (whole or in parts, also one that keeps no tile), every partial slot belongs to
// one unit, MM-DiT plans list their whole units longest first, and the per-XCD
// workgroup counts fit the grid. Prints one line per shape:
// "<name> units U whole W parts P slots S table 0|1 short C", C the units cut into
// parts whose query block holds at most 32 rows. It also checks the kernel's order of
// the units within a share when every segment ends on a short block.
#include <cstdio>
#include <cstdlib>
#include <initializer_list>
#include <map>
#include <vector>

#include "host_internal.h"
#include "tile_attn.h"
#include "unit_order.h"

using namespace ta::host;

namespace {

int check(const char* name, int B, int H, int F, int T, int P, int d, int g, int form, int hole = 0) {
  const int rows = d == 128 ? 128 : 256, slots_x = 64;
  std::vector<uint8_t> m((size_t)F * F);
  tile_attn_make_mask(F, g, form, m.data());
  if (hole > 0)  // query frames hole - 1, 2 hole - 1, ... keep nothing
    for (int i = hole - 1; i < F; i += hole)
      for (int j = 0; j < F; ++j) m[(size_t)i * F + j] = 0;
  int n_seg = F;
  std::vector<uint8_t> aug;
  if (P > 0) {  // the text row and column are kept entirely
    n_seg = F + 1;
    aug.assign((size_t)n_seg * n_seg, 1);
    for (int i = 0; i < F; ++i)
      for (int j = 0; j < F; ++j) aug[i * n_seg + j] = m[i * F + j];
  }
  HostWorkList hw = build_work_list(P > 0 ? aug.data() : m.data(), 1, H, n_seg, true);
  const int L = T > P ? T : P, nqb = (L + rows - 1) / rows;
  // as the forward does: the MM-DiT form runs each XCD's share longest first
  append_fwd_schedule(hw, B, nqb, rows, d, T, P, F, slots_x, true, P > 0);
  const int32_t* w = hw.words.data();
  const int32_t* items = w;
  const int32_t* cols = w + hw.off_cols;
  const int32_t* xcd = w + hw.off_xcd;
  const int32_t* pieces = w + hw.off_pieces;
  const int32_t* cut = w + hw.off_cut_units;
  if (hw.off_pieces != hw.off_xcd + 32) return std::printf("%s: pieces do not follow the XCD table\n", name), 1;
  const long per_b = (long)hw.n_items * nqb, n = B * per_b;
  const int tpf = (T + 63) / 64, ptiles = (P + 63) / 64;
  auto tiles = [&](long u) -> long {
    const int32_t* it = items + 5 * ((u % per_b) / nqb);
    const int qb = (int)(u % nqb), frame = it[1], beg = it[2], cnt = it[3];
    const int seg_len = (P > 0 && frame == F) ? P : T;
    if ((long)qb * rows >= seg_len) return 0;
    long t = (long)cnt * tpf;
    if (P > 0 && cnt > 0 && cols[beg + cnt - 1] == F) t += ptiles - tpf;
    return t;
  };
  auto has_rows = [&](long u) {
    const int32_t* it = items + 5 * ((u % per_b) / nqb);
    return (long)(u % nqb) * rows < ((P > 0 && it[1] == F) ? P : T);
  };
  std::vector<long> covered(n, 0), whole_runs(n, 0), part_runs(n, 0);
  std::map<int, int> slot_unit;
  long whole = 0, parts = 0;
  if (hw.unit_table && P == 0) return std::printf("%s: unit table without a text prefix\n", name), 1;
  for (int x = 0; x < 8; ++x) {
    if (xcd[4 * x + 1] + xcd[4 * x + 2] > hw.wg_per_xcd) return std::printf("%s: grid too small\n", name), 1;
    if (hw.unit_table && xcd[4 * x + 1] != 0) return std::printf("%s: contiguous units in a table plan\n", name), 1;
    for (int p = 0; p < xcd[4 * x + 1]; ++p) {
      covered[xcd[4 * x] + p] += tiles(xcd[4 * x] + p);
      ++whole_runs[xcd[4 * x] + p];
    }
    whole += xcd[4 * x + 1];
    long prev_len = -1;  // table entries of whole units come longest first
    for (int p = 0; p < xcd[4 * x + 2]; ++p) {
      const int32_t* pc = pieces + 4 * (xcd[4 * x + 3] + p);
      if (pc[0] < 0 || pc[0] >= n) return std::printf("%s: unit out of range\n", name), 1;
      if (pc[3] < 0) {  // a whole unit (possibly with no kept tile: its rows are still written)
        if (pc[1] != 0 || pc[2] != tiles(pc[0]) || !has_rows(pc[0])) return std::printf("%s: bad whole entry\n", name), 1;
        if (hw.unit_table && prev_len >= 0 && pc[2] > prev_len && part_runs[pc[0]] == 0)
          return std::printf("%s: table not longest first\n", name), 1;
        prev_len = pc[2];
        ++whole_runs[pc[0]];
        ++whole;
      } else {
        if (pc[1] < 0 || pc[2] <= 0 || pc[1] + pc[2] > tiles(pc[0])) return std::printf("%s: bad part\n", name), 1;
        if (!slot_unit.emplace(pc[3], pc[0]).second) return std::printf("%s: slot reused\n", name), 1;
        ++part_runs[pc[0]];
        ++parts;
      }
      covered[pc[0]] += pc[2];
    }
  }
  for (long u = 0; u < n; ++u) {
    if (covered[u] != tiles(u)) return std::printf("%s: unit %ld covers %ld of %ld tiles\n", name, u, covered[u], tiles(u)), 1;
    // every unit with rows runs exactly once, whole or in parts; one without rows at most
    // as a contiguous whole unit (the kernel returns at once)
    const bool once = (whole_runs[u] == 1 && part_runs[u] == 0) || (whole_runs[u] == 0 && part_runs[u] > 0);
    if (has_rows(u) ? !once : (part_runs[u] > 0 || whole_runs[u] > 1))
      return std::printf("%s: unit %ld runs %ld whole and %ld parts\n", name, u, whole_runs[u], part_runs[u]), 1;
  }
  int slots = 0;
  for (int k = 0; k < hw.n_cut_units; ++k)
    for (int s = cut[3 * k + 1]; s < cut[3 * k + 1] + cut[3 * k + 2]; ++s, ++slots)
      if (slot_unit.count(s) == 0 || slot_unit[s] != cut[3 * k]) return std::printf("%s: slot of another unit\n", name), 1;
  if (slots != hw.n_part_slots || (int)slot_unit.size() != hw.n_part_slots) return std::printf("%s: slot count\n", name), 1;
  int cut_short = 0;  // units cut into parts whose query block holds at most 32 rows
  for (int k = 0; k < hw.n_cut_units; ++k) {
    const int32_t* it = items + 5 * ((cut[3 * k] % per_b) / nqb);
    const int seg_len = (P > 0 && it[1] == F) ? P : T;
    if (seg_len - (int)(cut[3 * k] % nqb) * rows <= 32) ++cut_short;
  }
  std::printf("%s units %ld whole %ld parts %ld slots %d table %d short %d\n", name, n, whole, parts,
              hw.n_part_slots, (int)hw.unit_table, cut_short);
  return 0;
}

// The kernel's order of a share whose segments all end on a short block
// (ta::short_last_unit): every position maps to a distinct unit of the share, the
// full blocks come first and the short ones last, each in their original order.
int check_short_last(uint32_t n_items, uint32_t nqb) {
  const uint32_t n = n_items * nqb;
  for (uint32_t x = 0; x < 8; ++x) {
    const uint32_t s = ta::share_start(n, x), cnt = ta::share_count(n, x);
    std::vector<int> seen(cnt, 0);
    long prev_full = -1, prev_short = -1;
    bool in_short = false;
    for (uint32_t pos = 0; pos < cnt; ++pos) {
      const uint32_t u = ta::short_last_unit(n, nqb, x, pos);
      if (u < s || u >= s + cnt || seen[u - s]++) return std::printf("short-last %u %u: bad unit\n", n_items, nqb), 1;
      const bool is_short = u % nqb == nqb - 1;
      if (in_short && !is_short) return std::printf("short-last %u %u: full after short\n", n_items, nqb), 1;
      in_short = is_short;
      long& prev = is_short ? prev_short : prev_full;
      if ((long)u <= prev) return std::printf("short-last %u %u: order\n", n_items, nqb), 1;
      prev = (long)u;
    }
  }
  return 0;
}

}  // namespace

int main() {
  int bad = 0;
  bad |= check("93f-col", 1, 24, 24, 3600, 0, 96, 1, TA_MASK_COL);
  bad |= check("29f-col", 1, 24, 8, 3600, 0, 96, 1, TA_MASK_COL);
  bad |= check("sp-col", 1, 6, 24, 3600, 0, 96, 1, TA_MASK_COL);
  bad |= check("sp-sym", 1, 6, 24, 3600, 0, 96, 1, TA_MASK_SYM);
  bad |= check("long-col", 1, 24, 48, 1200, 0, 96, 2, TA_MASK_COL);
  bad |= check("d128-sym", 1, 18, 24, 3600, 0, 128, 1, TA_MASK_SYM);
  bad |= check("cog-sym", 1, 48, 13, 1350, 226, 64, 1, TA_MASK_SYM);
  bad |= check("cog-sym2", 1, 48, 13, 1350, 226, 64, 2, TA_MASK_SYM);
  bad |= check("batch3", 3, 5, 7, 333, 0, 96, 2, TA_MASK_SYM);
  // the shapes of test_ragged_round_in_parts (tests/test_gpu_parity.py, and gpu-e in
  // tests/test_gpu_mmdit.py)
  bad |= check("gpu-a", 1, 16, 17, 500, 0, 64, 1, TA_MASK_COL);
  bad |= check("gpu-b", 1, 12, 20, 700, 0, 96, 2, TA_MASK_COL);
  bad |= check("gpu-c", 1, 32, 6, 700, 0, 96, 1, TA_MASK_SYM);
  bad |= check("gpu-d", 1, 8, 11, 700, 0, 128, 1, TA_MASK_COL);
  bad |= check("gpu-e", 1, 12, 9, 1350, 226, 64, 1, TA_MASK_SYM);
  // query frames that keep nothing, some of them in the ragged round cut into parts
  bad |= check("gpu-f", 1, 12, 20, 700, 0, 96, 2, TA_MASK_COL, 7);
  // short last query blocks (16 rows): at d = 64 run last, no parts; at d = 128 among
  // the units cut into parts
  bad |= check("gpu-g", 1, 32, 6, 528, 0, 64, 1, TA_MASK_COL);
  bad |= check("gpu-h", 1, 20, 6, 528, 0, 128, 1, TA_MASK_COL);
  int orders = 0;
  for (uint32_t nqb : {2u, 3u, 15u, 29u})
    for (uint32_t items : {1u, 3u, 7u, 8u, 9u, 57u, 576u, 1153u}) {
      bad |= check_short_last(items, nqb);
      ++orders;
    }
  std::printf("short-last orders %d\n", orders);
  return bad;
}

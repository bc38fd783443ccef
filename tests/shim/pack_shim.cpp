// Test-only host shim: exposes the library's genome packer without any GPU so the CPU test suite
// can interpret packed programs and compare them with the oracle.
#include <cstring>
#include <string>
#include <vector>

#include "../../paper_2608_27612_amd/csrc/pack.h"

extern "C" int shim_pack(const emr_genome* g, uint32_t* blob, int64_t blob_cap, int64_t* blob_words,
                         uint32_t* desc8, int32_t* info_out, char* msg, int msg_cap) {
  std::vector<uint32_t> b;
  emr::ProgDesc d[2];
  emr::GenomeInfo inf[2];
  emr_status st = EMR_OK;
  std::string m;
  if (!emr::pack_genome(*g, b, d, inf, &st, &m)) {
    std::strncpy(msg, m.c_str(), (size_t)msg_cap - 1);
    msg[msg_cap - 1] = 0;
    return (int)st;
  }
  *blob_words = (int64_t)b.size();
  if ((int64_t)b.size() > blob_cap) return 1;
  std::memcpy(blob, b.data(), b.size() * 4);
  for (int k = 0; k < 2; ++k) {
    desc8[8 * k + 0] = d[k].var_off;
    desc8[8 * k + 1] = d[k].n_rec;
    desc8[8 * k + 2] = d[k].n_steps;
    desc8[8 * k + 3] = d[k].uni_off;
    desc8[8 * k + 4] = d[k].flags;
    desc8[8 * k + 5] = d[k].uni_end;
    int32_t* o = info_out + 12 * k;
    o[0] = inf[k].n_steps; o[1] = inf[k].fma_xy; o[2] = inf[k].fma_node;
    for (int a = 0; a < 6; ++a) o[3 + a] = inf[k].act_count[a];
    o[9] = inf[k].window; o[10] = inf[k].n_unodes; o[11] = inf[k].out_varying ? 1 : 0;
  }
  return 0;
}

// The compiled tier's host side: one program's machine words and listing.
#include "../../paper_2608_27612_amd/csrc/jit.h"

extern "C" int shim_compile(const uint32_t* rec, uint32_t n_rec, int output_varies, int S, int P,
                            int W, uint32_t* words, int64_t cap, int64_t* n_words, char* listing,
                            int64_t listing_cap, char* msg, int msg_cap) {
  emr::jit::Code code;
  std::string m;
  if (!emr::jit::compile_program(rec, n_rec, output_varies != 0, S, P, W, true, &code, &m)) {
    std::strncpy(msg, m.c_str(), (size_t)msg_cap - 1);
    msg[msg_cap - 1] = 0;
    return 1;
  }
  *n_words = (int64_t)code.words.size();
  if ((int64_t)code.words.size() > cap || (int64_t)code.listing.size() + 1 > listing_cap) return 2;
  std::memcpy(words, code.words.data(), code.words.size() * 4);
  std::memcpy(listing, code.listing.c_str(), code.listing.size() + 1);
  return 0;
}

// The template code object with its code area grown to new_bytes; *area_off: the area's file offset.
extern "C" int shim_grow(const uint8_t* img, int64_t n, int64_t area_bytes, int64_t new_bytes,
                         uint8_t* out, int64_t cap, int64_t* n_out, int64_t* area_off, char* msg,
                         int msg_cap) {
  emr::jit::AreaInfo info;
  std::string m;
  std::vector<uint8_t> o;
  if (!emr::jit::find_area(img, (size_t)n, (size_t)area_bytes, &info, &m) ||
      !emr::jit::grow_area(img, (size_t)n, info, (size_t)new_bytes, &o, &m)) {
    std::strncpy(msg, m.c_str(), (size_t)msg_cap - 1);
    msg[msg_cap - 1] = 0;
    return 1;
  }
  *n_out = (int64_t)o.size();
  *area_off = (int64_t)info.file_off;
  if ((int64_t)o.size() > cap) return 2;
  std::memcpy(out, o.data(), o.size());
  return 0;
}

// A population's packing and a call's plan, built on the host exactly as the library builds them
// (packing in n_parts ranges, as threads do), then checked with the library's table check. With
// plant > 0 one entry is made wrong before the check (1: a group's bias rows past the table, 2: a
// group's pair past the call, 3: a member's source past the sources, 4: a descriptor's records
// past the program words, 5: one pair in two groups, 6: the workspace totals over the pool).
// Returns 0 when the tables check out, 1 when the check refuses them, else the build's status;
// stats[0..4]: groups, members, bias floats, program words, buckets.
#include "../../paper_2608_27612_amd/csrc/plan.h"

extern "C" int shim_plan_check(const emr_genome* genomes, int32_t n_genomes, int n_parts,
                               const emr_source* sources, int32_t n_sources, const int32_t* offs,
                               int32_t n_shared, int32_t depth, int plant, int64_t* stats,
                               char* msg, int msg_cap) {
  auto put = [&](const std::string& m) {
    std::strncpy(msg, m.c_str(), (size_t)msg_cap - 1);
    msg[msg_cap - 1] = 0;
  };
  std::vector<emr::ProgDesc> desc;
  std::vector<emr::GenomeInfo> info;
  std::vector<uint32_t> words;
  std::string m;
  int32_t bad = -1;
  emr_status st = emr::pack_genomes(
      n_genomes, [&](int32_t g) { return genomes[g]; }, n_parts,
      [](int k, const std::function<void(int)>& f) {
        for (int t = 0; t < k; ++t) f(t);
      },
      &desc, &info, &words, &bad, &m);
  if (st != EMR_OK) {
    put(m);
    return (int)st;
  }
  emr::PlanTables P;
  st = emr::build_plan_tables(desc.data(), info.data(), n_genomes, sources, n_sources, offs,
                              n_shared, depth, &P, &m);
  if (st != EMR_OK) {
    put(m);
    return (int)st;
  }
  stats[0] = (int64_t)P.groups.size();
  stats[1] = (int64_t)P.members.size();
  stats[2] = (int64_t)P.bias_floats;
  stats[3] = (int64_t)words.size();
  stats[4] = (int64_t)P.buckets.size();
  if (plant > 0 && P.groups.empty()) {
    put("nothing to plant in");
    return 2;
  }
  switch (plant) {
    case 1: P.groups.back().bias_off = (uint32_t)P.bias_floats; break;
    case 2: P.groups[0].pair[0] = (uint32_t)P.n_pairs; break;
    case 3: P.members.back().source = (uint32_t)n_sources; break;
    case 4: desc[P.members[0].desc].var_off = (uint32_t)words.size(); break;
    case 5:
      if (P.groups.size() < 2) {
        put("one group only");
        return 2;
      }
      P.groups[1].pair[0] = P.groups[0].pair[0];
      break;
    case 6: P.total = P.off_ptotal; break;
    default: break;
  }
  if (!emr::check_plan_tables(P, desc.data(), words.size(), &m)) {
    put(m);
    return 1;
  }
  put("ok");
  return 0;
}

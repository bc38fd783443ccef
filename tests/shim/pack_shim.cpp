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

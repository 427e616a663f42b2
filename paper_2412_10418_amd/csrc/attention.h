// Internal interface of the attention kernels (attention.hip).
#pragma once
#include "common.h"

namespace cdsl {

struct AttnArgs {
  PassDesc p;
  const float* Q;         // [M][H][hd] fp32, rotary already applied
  float* O;               // [M][H][hd] fp32 output (fp32 models)
  bf16* Ohi;              // [M][H][hd] hi / lo planes (bf16-weight models)
  bf16* Olo;
  KVPool pool;            // fp32 format (fp32 models) or split bf16 planes
  int layer;
  int H, Hkv, G;
  long long rows_total;   // M * H
  float scale_log2;       // log2(e) / sqrt(hd)
  float* part_o;          // [nsplit][M*H][hd]
  float* part_ml;         // [nsplit][M*H][2]  (running max in log2 units, sum)
  int nsplit, blocks_per_split;
};

// key blocks one workgroup (one key split) handles at most
constexpr int kAttnMaxList = 256;
// key splits of one pass at most
constexpr int kAttnMaxSplits = 16;

struct AttnPlan {
  int row_tiles, row_groups, threads;
  int kw;                 // key groups per row tile (1, 2 or 4)
  int nsplit, blocks_per_split;
};

// max_prefix_len: the longest prefix of the prompts in the pass (host copy).
AttnPlan attn_plan(const PassDesc& p, int H, int Hkv, int hd, int dtype, int max_prefix_len, int max_splits);
hipError_t attn_launch(const AttnArgs& a, const AttnPlan& pl, int hd, int dtype, hipStream_t st);
// the merge of split partials (a no-op when pl.nsplit == 1)
hipError_t attn_combine_launch(const AttnArgs& a, const AttnPlan& pl, int hd, hipStream_t st);

}  // namespace cdsl

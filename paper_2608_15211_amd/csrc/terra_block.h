// terra_block.h - argument blocks of the Swin-block kernels (block.hip),
// filled by the C ABI (abi.hip) from the public structs field by field.
#pragma once

namespace terra {

struct BlockParams {
  const float *ln1_g, *ln1_b;
  const void* w_qkv;
  const float* b_qkv;
  const void* w_proj;
  const float* b_proj;
  const float *ln2_g, *ln2_b;
  const void* w_fc1;
  const float* b_fc1;
  const void* w_fc2;
  const float* b_fc2;
};

struct BlockGrads {
  float *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_proj, *b_proj, *ln2_g, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
};

struct BlockSaved {
  float *mu1, *rstd1, *mu2, *rstd2;
  void *q, *k, *v, *o;
  float* lse;
  void* x1;
  void *h, *a;
};

}  // namespace terra

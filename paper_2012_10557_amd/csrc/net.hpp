// ResNet18 edge classifier as a fixed table of layers.
//
// Topology: He et al., "Deep residual learning for image recognition" (the
// paper's ResNet reference), torchvision's ResNet18: a 7x7/2 stem conv with
// BatchNorm, ReLU and 3x3/2 max pooling; four stages of two BasicBlocks
// (widths 64/128/256/512, stride 2 entering stages 2-4 with a 1x1/2
// projection shortcut); global average pooling; an affine classifier, or
// (hidden > 0, the number of neurons in the last layer that retraining
// configurations vary, sections 3.2 and 6.1) a hidden fully connected ReLU
// layer of `hidden` neurons and then the classifier.
// Stages (the unit of freezing, section 3.1): 0 stem, 1-4 layer1-4, 5 fc.
//
// Parameter offsets follow the canonical flat layout (torchvision state_dict
// order without num_batches_tracked).  Inside the library conv weights sit at
// the same offsets but permuted to [K][R][S][C] ("internal layout").
#pragma once

#include <stdint.h>

#include <vector>

namespace ekya {

struct ConvL {
  int cin, cout, R, S, stride, pad, stage;
  long long off;       // parameter offset (fp32 master)
  int bn;              // BatchNorm following this conv
  int cin_pad;         // stored input channels (stem: padded to the 16-byte unit)
  long long sh_krsc;   // shadow offset (elements) of [K][R][S][cin_pad]
  long long sh_crsk;   // shadow offset of [C][R][S][K] (-1 for the stem)
};

struct BnL {
  int C, stage;
  long long g, b, rm, rv;  // parameter offsets
  long long st;            // offset into per-channel scratch (sum of earlier C)
};

struct BlockL {
  int c1, c2, cd;  // conv indices (cd = -1: identity shortcut)
  int stage;
};

struct Net {
  int n_classes = 0;
  int dt = 0;
  std::vector<ConvL> conv;
  std::vector<BnL> bn;
  std::vector<BlockL> blk;
  int hidden = 0;                    // neurons of the hidden classifier layer (0: none)
  long long fc1_w = -1, fc1_b = -1;  // hidden layer [hidden][512], [hidden]
  long long fc_w = 0, fc_b = 0, total = 0;  // output layer [classes][head_in()], [classes]
  long long stage_begin[7] = {0};  // first parameter offset of each stage; [6] = total
  long long bn_channels = 0;       // sum of C over all BatchNorm layers
  long long shadow_elems = 0;
  int widths[4] = {64, 128, 256, 512};

  static Net build(int n_classes, int dt, int hidden = 0);
  int head_in() const { return hidden > 0 ? hidden : 512; }

  // Host tables for the kernels (see kernels.hpp for row formats).
  std::vector<long long> permute_table() const;              // every tensor
  std::vector<long long> fold_table(int lo_stage, int hi_stage) const;  // BNs of stages
  std::vector<long long> pack_table(int lo_stage, int hi_stage, bool with_crsk) const;
};

// Spatial sizes for one input resolution.
struct Geo {
  int H = 0, W = 0;
  std::vector<int> ih, iw, oh, ow;  // per conv: input and output spatial size
  int sh = 0, sw = 0;               // stem conv output
  int mh = 0, mw = 0;               // max-pool output (input of layer1)
  int lh[5] = {0}, lw[5] = {0};     // output of layer i (1..4)

  static Geo build(const Net& net, int H, int W);
  // Elements per frame of the input of stage s (s = 0: padded frame; s = 5:
  // the pooled 512 features, stored as fp32).
  long long stage_in_elems(const Net& net, int s) const;
  int stage_in_channels(const Net& net, int s) const;
};

}  // namespace ekya

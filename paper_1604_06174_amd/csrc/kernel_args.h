// By-value argument blocks of the fp32 convolution and GEMM kernels (shared
// by their sources and by the host-only launch checker, which reads their
// pointer fields).
#pragma once

namespace ckpt {

struct ConvArgs {
  const float *X;   // kernel input  [N, Hx, Wx, C]
  const float *Wt;  // weights [Cout, 3, 3, Cin]
  float *Y;         // kernel output [N, H, W, J]
  int N, H, W;      // output dims
  int Hx, Wx;       // input dims
  int C, J;         // reduction / output channels
  int R, rblk;      // output rows per workgroup, workgroups per image
  const float *E0, *E1;  // epilogue operands (MASK: E0; SC: E0 = g, E1 = y)
  int Eh, Ew, Ec;        // SC2: dims of g and y
  double *stats;         // STATS: [2][J][gridDim.x] (sum v, sum v^2; channel-major)
  const float *tst, *tg, *tb;  // optional bn_relu: FWD input / DGRAD MASK transform
  float *rout;  // FWD, stride 1, with tst: the transformed input rows the workgroup owns
};

struct WgArgs {
  const float *X;   // conv input [N, Hx, Wx, C]
  const float *DY;  // conv output gradient [N, H, W, J]
  float *part;      // [gridDim.x][J][9C]
  int N, H, W, Hx, Wx, C, J, S;
  int pix_per_blk;  // multiple of WG_KC
  const float *tst, *tg, *tb;  // optional bn_relu of the input X
};

struct GemmArgs {
  int M, N, K;
  const float *A;
  int lda;
  const float *B;
  int ldb;
  float *C;
  int ldc;
  const float *D;  // ADD
  int ldd;
  const float *bias;  // MLPFWD
  float *Z;           // MLPFWD
  int ldz;
};

}  // namespace ckpt

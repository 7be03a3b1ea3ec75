// pc_replay_hybrid.hip -- the hybrid-layout replay kernel (block keys,
// prefix ids and the S3-FIFO ghost table in global memory, the rest of the
// state in LDS, two instances per CU) in a translation unit of its own, so
// that it is built under its own machine scheduler (build.py).
#define PC_REPLAY_HYBRID_TU 1
#include "pc_replay.hip"

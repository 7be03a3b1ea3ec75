// pc_replay_global.hip -- the replay kernels whose state is partly or wholly
// in global memory (hybrid layout: block keys, prefix ids and the S3-FIFO
// ghost table; workspace layout: everything), two instances per CU, in a
// translation unit of their own, so that they are built under their own
// machine scheduler (build.py).
#define PC_REPLAY_GLOBAL_TU 1
#include "pc_replay.hip"

// The eight-wave decode kernels (small batches at short contexts, where each
// wave of a four-wave workgroup would stream at most four chunks): the same
// source as decode.hip, compiled apart so that the two kernel sets build in
// parallel. Only the eight-wave dispatch chain and its kernels come from here;
// planning, the fixed scratch array and the four-wave kernels stay in decode.hip.
#define TK_DECODE_SHORT_UNIT 1
#include "decode.hip"

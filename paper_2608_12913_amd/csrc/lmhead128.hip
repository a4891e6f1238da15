// The streaming LM-head kernel with 128 rows per workgroup (used above 64 rows
// when the many-row kernel does not apply): the source of lmhead.hip compiled with
// that row shape.
#define DCD_STREAM_ROWS 128
#include "lmhead.hip"

// Device translation unit of the PuzzleKV library: every kernel of the hot
// path for gfx950, compiled as one unit so the sticky status word is shared.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <mutex>
#include <type_traits>

#include "pkv_internal.h"

#include "cache_ops.inl"
#include "int4.inl"
#include "compress.inl"
#include "compress_qr.inl"
#include "attention.inl"
#include "attention_mfma.inl"
#include "attention_launch.inl"
#include "global_svd.inl"
#include "bandwidth.inl"

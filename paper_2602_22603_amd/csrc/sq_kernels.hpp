// sq_kernels.hpp - everything the host library (store.cpp) needs from the
// gfx950 kernel files: constants, pool layout, kernel arguments, launchers.
// Internal to libsq.
#pragma once

#include "decode_args.hpp"
#include "extend_args.hpp"
#include "kv_args.hpp"
#include "sq_common.hpp"

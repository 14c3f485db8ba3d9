// fallback.hip built for the host emulation as its own translation unit (the
// emulator's globals live in screen_i8_host.cpp).
#include "hip/hip_runtime.h"
#include "fallback_host_src.hip"

// Host build of libsalt for tests: see hip_runtime.h.
#pragma once
#include "hip_runtime.h"

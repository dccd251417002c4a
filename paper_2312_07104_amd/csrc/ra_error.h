// Per-thread error text behind ra_last_error().
#pragma once
#include <string>

#include "radixattn.h"

int ra_fail(int code, const std::string& msg);
int ra_ok();

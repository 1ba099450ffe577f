/* Thread-local error reporting shared by the C and C++ sources of liblaser. */
#ifndef LASER_ERROR_H
#define LASER_ERROR_H

#include "laser.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Records a printf-style message for laser_last_error() and returns `code`. */
laser_status laser_fail(laser_status code, const char* fmt, ...);
void laser_clear_error(void);

#ifdef __cplusplus
}
#endif
#endif

// Library-wide entry points: error text and version.
#include "cel_internal.h"

namespace cel {
const char *last_error_text();
}

extern "C" const char *cel_last_error(void) { return cel::last_error_text(); }

extern "C" int cel_version(void) { return 100; /* 0.1.0 */ }

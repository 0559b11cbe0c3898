/* The status strings as a C caller sees them: any int is a valid
 * park_status argument in C, including values outside the enumerators. */
#include <stddef.h>
#include <string.h>

#include "park.h"

int host_check_status_strings(void) {
  int bad = 0;
  for (int s = -3; s < 120; ++s) {
    const char* m = park_status_string((park_status)s);
    if (m == NULL) ++bad;
    else if ((s < 0 || s > 5) && strcmp(m, "unknown status") != 0) ++bad;
  }
  return bad;
}

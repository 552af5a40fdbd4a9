"""MI355X-native shared KV-cache pool with batched paged decode attention.

The native library is ``libcrosspool.so`` (C ABI in include/crosspool.h);
``paper_2606_24506_amd.crosspool`` is its ctypes binding. Importing the
package itself loads nothing, so the build step can import it before the
library exists.
"""

__all__ = ["crosspool", "build"]

"""Location of the built HIP library (kept separate so nothing loads it by accident)."""
import os

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libmasq.so")

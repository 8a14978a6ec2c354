"""CPU oracle for the Taliesin KV save/verify/restore path.

TEST INFRASTRUCTURE ONLY. Nothing in the product package may import this
package; only tests, the smoke check and the benchmark's CPU baseline use it.
It shares no code with the HIP path. See taliesin_ref for the definitions.
"""
from .taliesin_ref import *  # noqa: F401,F403

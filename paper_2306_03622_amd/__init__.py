"""Pipelined model swap-in and execution on one AMD MI355X (libtorpor + ctypes binding)."""
from .torpor import *  # noqa: F401,F403
from .torpor import Runtime, ModelDesc, TorporError, HostArena, lib, host_lib  # noqa: F401

"""MI355X (gfx950) paged grouped-query decode attention."""
